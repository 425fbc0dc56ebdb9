"""GPU parity on the five workloads at full size, in the launch configuration
the benchmark times.  Every op of each layer stack is compared with the
oracle fed the GPU's own input to that op: structures bit-exact, pool/unpool
copies exact, convolutions on sampled rows (every leaf size included) within
1e-5 + 1e-4 |oracle|.
"""
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
    from paper_1611_05009_amd import octnet
    octnet.lib()


def host(t):
    return t.detach().cpu().numpy()


def ref_grid(g):
    return O.make_grid(trees_np(g.trees), *g.dims())


def check_structure(g, ref):
    assert g.dims() == (ref.n, ref.gd, ref.gh, ref.gw)
    assert np.array_equal(trees_np(g.trees), ref.trees)
    assert np.array_equal(host(g.prefix), ref.prefix)


@pytest.mark.parametrize("key", ["c1", "c2", "c3", "c4", "c5"])
def test_workload_chain(key):
    from paper_1611_05009_amd import pipeline
    log("workload %s: generating inputs" % key)
    W = pipeline.Workload(key)
    recs = []
    pipeline.run_step(W, recs)
    torch.cuda.synchronize()
    log("workload %s: %d leaves, %d ops" % (key, W.n_leaves, len(recs)))
    for k, r in enumerate(recs):
        log("  op %d %s" % (k, r.op))
        if r.op == "input":
            ref = O.build(W.occ_np)
            check_structure(r.g_out, ref)
            if W.dense is not None:
                want = O.ten2oc(ref, W.dense.cpu().numpy(), "avg")
                assert_close(host(r.x_out), want, "%s ten2oc" % key)
            continue
        gi = ref_grid(r.g_in)
        xi = host(r.x_in)
        if r.op == "conv":
            info = O.leaf_info(gi)
            rows = sample_rows(gi.n_leaves, info, 1500, seed=k)
            p = r.params
            want = O.conv3_sampled(gi, xi, host(p["w"]), host(p["b"]), p["relu"], rows, info=info)
            assert_close(host(r.x_out)[rows], want, "%s op %d conv" % (key, k))
        elif r.op == "pool":
            go = O.pool2_structure(gi)
            check_structure(r.g_out, go)
            out = host(r.x_out)
            rows = sample_rows(go.n_leaves, O.leaf_info(go), 20000, seed=k)
            _, want = O.pool2_max(gi, xi, go, rows=rows)
            assert np.array_equal(out[rows], want.astype(np.float32))
        elif r.op in ("unpool", "unpool_guided"):
            if r.op == "unpool":
                go = O.unpool2_structure(gi)
            else:
                go = ref_grid(r.g_out)  # the guide; its pooling must be the input
                assert np.array_equal(O.pool2_structure(go).trees, gi.trees)
            check_structure(r.g_out, go)
            rows = sample_rows(go.n_leaves, O.leaf_info(go), 20000, seed=k)
            _, want = O.unpool2(gi, xi, guide=go if r.op == "unpool_guided" else None, rows=rows)
            assert np.array_equal(host(r.x_out)[rows], want.astype(np.float32))
        else:
            raise AssertionError(r.op)
