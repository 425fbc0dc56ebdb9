"""oc_build_noalloc (the entry point for callers that cannot allocate: its
scratch is a static device array) against oc_build, bit for bit: two calls
in a row on the same device, the second on a smaller input, so that the
array's contents from the first call must not leak into the second."""
import numpy as np
import pytest
import torch

from common import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_build_noalloc_matches_build_twice():
    from paper_1611_05009_amd import octnet as oc
    rng = np.random.default_rng(77)
    for k, (n, gd, gh, gw, p) in enumerate([(3, 12, 10, 9, 0.03), (1, 4, 5, 3, 0.2)]):
        occ = (rng.random((n, 8 * gd, 8 * gh, 8 * gw)) < p).astype(np.uint8)
        # a solid block as well, so that both split rules differ
        occ[0, 8:24, 8:16, 0:16] = 1
        dev = torch.from_numpy(occ).cuda()
        for rule in ("mixed", "any"):
            want = oc.build(dev, rule)
            got = oc.build_noalloc(dev, rule)
            torch.cuda.synchronize()
            log("call %d rule %s: %d trees, %d leaves" % (k, rule, want.n_trees, want.n_leaves))
            assert got.n_leaves == want.n_leaves
            assert torch.equal(got.trees, want.trees)
            assert torch.equal(got.prefix, want.prefix)


def test_build_noalloc_rejects_too_many_trees():
    import ctypes
    from paper_1611_05009_amd import octnet as oc
    nl = ctypes.c_int64(0)
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the size check comes first
    rc = oc.lib().oc_build_noalloc(fake, 1, 256, 128, 129, 0, fake, fake, ctypes.byref(nl), None)
    assert rc == oc.lib().oc_build_noalloc(fake, 9, 128, 64, 64, 0, fake, fake, ctypes.byref(nl), None) == -5
    assert b"static scratch" in oc.lib().oc_last_error()
