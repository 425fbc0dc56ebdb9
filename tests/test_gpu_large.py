"""The fused convolution past 4 GiB of input: ten 256^3 samples of 2%
uniform noise give about 38 M leaves, so with 32 channels the input rows
extend past byte 2^32.  The fused kernels address rows by a 32-bit row
index (structured buffer loads) and must not fall back or wrap there.
Sampled rows of the first sample and of the last one (whose rows all lie
past byte 2^32), every leaf size included, are compared with the oracle
run on that sample alone (samples do not interact)."""
import numpy as np
import pytest
import torch

import octref as O
from common import assert_close, log, sample_rows, trees_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_conv_past_4gib_of_input():
    from paper_1611_05009_amd import octnet as oc
    rng = np.random.default_rng(4242)
    n, res = 10, 256
    occ = np.empty((n, res, res, res), dtype=np.uint8)
    for s in range(n):
        occ[s] = rng.random((res, res, res), dtype=np.float32) < 0.02
    g = oc.build(torch.from_numpy(occ).cuda())
    log("noise 256^3 x %d: %d leaves, input %.2f GiB" % (n, g.n_leaves, g.n_leaves * 128 / 2**30))
    assert g.n_leaves * 32 * 4 > 2**32
    assert oc.mfma_supported(32, 32)
    gen = torch.Generator(device="cuda").manual_seed(5)
    x = torch.randn((g.n_leaves, 32), generator=gen, device="cuda", dtype=torch.float32)
    w = (rng.standard_normal((32, 32, 3, 3, 3)) / np.sqrt(27 * 32)).astype(np.float32)
    b = rng.standard_normal(32).astype(np.float32)
    y = oc.conv3x3x3(g, x, torch.from_numpy(w).cuda(), torch.from_numpy(b).cuda(), impl="mfma")
    torch.cuda.synchronize()
    pre = g.prefix.cpu().numpy()
    per = g.gd * g.gh * g.gw
    trees = trees_np(g.trees)
    for s in (0, n - 1):
        a0, a1 = int(pre[s * per]), int(pre[(s + 1) * per])
        gs = O.make_grid(np.ascontiguousarray(trees[s * per:(s + 1) * per]), 1, g.gd, g.gh, g.gw)
        rows = sample_rows(a1 - a0, O.leaf_info(gs), 3000, seed=s)
        want = O.conv3(gs, x[a0:a1].cpu().numpy(), w, b, rows=rows)
        got = y[a0 + torch.from_numpy(rows).cuda()].cpu().numpy()
        log("  sample %d: rows %d..%d (byte %.2f GiB ..)" % (s, a0, a1, a0 * 128 / 2**30))
        if s == n - 1:
            assert a0 * 128 > 2**32
        assert_close(got, want, "conv past 4 GiB, sample %d" % s)
