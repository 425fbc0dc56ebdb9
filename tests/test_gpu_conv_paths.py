"""GPU parity of the convolution on random canonical split strings.

Drawing the split bits node by node puts cells of every size next to every
kind of neighbour: edge-8 cells beside split trees in all 26 directions,
edge-4 cells beside split depth-1 nodes (in their own tree and in the
neighbouring ones), edge-2 cells and unit voxels beside all of these, at the
grid boundary and inside.  The MFMA path (unit-voxel groups, boundary sums,
edge-8/4/2 cell kernels) is compared with the oracle element by element.
"""
import numpy as np
import pytest
import torch

import octref as O
from common import assert_close, log
from paper_1611_05009_amd import synth

pytestmark = pytest.mark.gpu

oc = None


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    global oc
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1611_05009_amd import octnet
    octnet.lib()
    oc = octnet
    torch.cuda.set_device(0)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


from test_conv_paths_cpu import CASES  # noqa: E402


@pytest.mark.parametrize("cin,cout", [(32, 32), (16, 32), (8, 16), (4, 16), (32, 8), (16, 4), (32, 2)])
@pytest.mark.parametrize("case", CASES)
def test_conv_random_split_strings(case, cin, cout):
    seed, n, gd, gh, gw, p0, p1, p2 = case
    rng = np.random.default_rng(seed)
    words = synth.random_trees(rng, n, gd, gh, gw, p0, p1, p2)
    ref = O.make_grid(words, n, gd, gh, gw)
    g = oc.from_trees(dev(words.view(np.int32)), n, gd, gh, gw)
    assert g.n_leaves == ref.n_leaves
    x = rng.standard_normal((ref.n_leaves, cin)).astype(np.float32)
    w = (rng.standard_normal((cout, cin, 3, 3, 3)) / np.sqrt(27 * cin)).astype(np.float32)
    b = rng.standard_normal(cout).astype(np.float32)
    log("case %s cin %d cout %d: %d leaves" % (case, cin, cout, ref.n_leaves))
    impl = "mfma" if oc.mfma_supported(cin, cout) else "generic"
    got = oc.conv3x3x3(g, dev(x), dev(w), dev(b), impl=impl).cpu().numpy()
    assert_close(got, O.conv3(ref, x, w, b), "conv %s %dx%d %s" % (impl, cin, cout, case))
