"""Workspace sized from the structure's own counts.

The exact query counts the boundary-sum slots (split trees plus split
depth-1 nodes, Sec. 3.1) on the device.  The count is checked against the
same count taken on the host from the bit strings, the size against the
host-only size-by-slots query, and a convolution run in the exact workspace
(and in one between the exact size and the bound) against the same
convolution in the bound-sized workspace, bit for bit: the layout changes,
the arithmetic does not.  One case is compared with the oracle as well.
"""
import ctypes

import numpy as np
import pytest
import torch

import octref as O
from common import assert_close, log, trees_np
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


def host_slots(words):
    w0 = words[:, 0].astype(np.int64)
    root = (w0 & 1) == 1
    d1 = np.zeros(len(w0), np.int64)
    for j in range(1, 9):
        d1 += (w0 >> j) & 1
    return int(root.sum() + d1[root].sum())


def slots_bytes(g, cin, cout, slots):
    nb = ctypes.c_size_t(0)
    assert oc.lib().oc_conv3x3x3_workspace_slots(g.n_trees, g.n_leaves, cin, cout, slots, ctypes.byref(nb)) == 0
    return nb.value


CASES = [  # seed, n, gd, gh, gw, p_root, p_d1, p_d2
    (1, 2, 3, 4, 5, 0.6, 0.5, 0.5),
    (2, 1, 4, 4, 4, 0.0, 0.5, 0.5),   # no split tree: one slot all the same
    (3, 1, 3, 3, 3, 1.0, 1.0, 1.0),   # every node split
    (4, 3, 5, 3, 4, 0.9, 0.3, 0.8),
]


@pytest.mark.parametrize("cin,cout", [(32, 32), (16, 32), (4, 16), (64, 64)])
@pytest.mark.parametrize("case", CASES)
def test_exact_workspace_matches_bound(case, cin, cout):
    seed, n, gd, gh, gw, p0, p1, p2 = case
    rng = np.random.default_rng(seed)
    words = synth.random_trees(rng, n, gd, gh, gw, p0, p1, p2)
    g = oc.from_trees(torch.from_numpy(words.view(np.int32)).cuda(), n, gd, gh, gw)
    slots = host_slots(words)
    exact = oc.conv_workspace_bytes(g, cin, cout)
    bound = oc.conv_workspace_bytes(g, cin, cout, exact=False)
    log("case %s %dx%d: %d leaves, %d slots, workspace %d (bound %d)" % (case, cin, cout, g.n_leaves, slots,
                                                                        exact, bound))
    assert exact == slots_bytes(g, cin, cout, slots)
    assert exact <= bound
    x = torch.from_numpy(rng.standard_normal((g.n_leaves, cin)).astype(np.float32)).cuda()
    w = torch.from_numpy((rng.standard_normal((cout, cin, 3, 3, 3)) / np.sqrt(27 * cin)).astype(np.float32)).cuda()
    b = torch.from_numpy(rng.standard_normal(cout).astype(np.float32)).cuda()
    outs = []
    for nbytes in sorted({exact, (exact + bound) // 2, bound}):
        # garbage in the workspace must not matter
        ws = torch.full((nbytes,), 0x7F, dtype=torch.uint8, device="cuda")
        outs.append(oc.conv3x3x3(g, x, w, b, relu=True, impl="mfma", ws=ws))
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    if case == CASES[0] and cin == 32:
        ref = O.make_grid(words, n, gd, gh, gw)
        assert_close(outs[0].cpu().numpy(), O.conv3(ref, x.cpu().numpy(), w.cpu().numpy(), b.cpu().numpy(), True),
                     "exact workspace vs oracle")


def test_exact_workspace_on_surfaces():
    """A 256^3 surface sample: far fewer slots than the bound counts."""
    from paper_1611_05009_amd import pipeline
    W = pipeline.Workload("c4")
    g = oc.build(W.occ)
    words = trees_np(g.trees)
    slots = host_slots(words)
    exact = oc.conv_workspace_bytes(g, 32, 32)
    bound = oc.conv_workspace_bytes(g, 32, 32, exact=False)
    log("c4: %d leaves, %d slots (bound %d), workspace %.2f GB (bound %.2f GB)"
        % (g.n_leaves, slots, (g.n_leaves - g.n_trees) // 7, exact / 1e9, bound / 1e9))
    assert exact == slots_bytes(g, 32, 32, slots)
    assert exact < bound
