"""Shared helpers for the GPU parity tests (inputs, comparisons)."""
from __future__ import annotations

import functools
import os
import sys

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_1611_05009_amd import synth  # noqa: E402

# Float parity bar: |gpu - oracle| <= ATOL + RTOL * |oracle|, element-wise, fp32.
RTOL = 1e-4
ATOL = 1e-5


def assert_close(got, want, what=""):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    err = np.abs(got - want)
    lim = ATOL + RTOL * np.abs(want)
    bad = err > lim
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError("%s: %d/%d elements out of tolerance; first at %s: got %r want %r"
                             % (what, int(bad.sum()), bad.size, tuple(i), got[tuple(i)], want[tuple(i)]))


# fp32 unit roundoff.  A sum of many terms evaluated in fp32, in any order,
# carries rounding errors on the scale of U32 * sum |terms| (one rounding of
# the largest partial sums); a dropped, doubled or misplaced term moves the
# result by a whole term, far above that scale.
U32 = 2.0 ** -24


def assert_close_sum(got, want, absum, what, k=1.0):
    """Bar for results that are sums over many leaves or voxels (gradients,
    the truncated-kernel conv): |got - want| <= ATOL + RTOL |want| +
    k U32 absum element-wise, absum >= sum |terms| (the oracle's same op on
    |inputs|).  The plain bar ATOL + RTOL |want| alone cannot hold where the
    sum cancels to |want| << absum: fp32 rounding of the terms alone leaves
    errors of that order.  Logs how many elements the plain bar misses."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    absum = np.asarray(absum, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    err = np.abs(got - want)
    plain = ATOL + RTOL * np.abs(want)
    lim = plain + k * U32 * absum
    n_plain = int((err > plain).sum())
    log("  %s: max err/bar %.3g (k=%g), plain bar missed by %d/%d (max ratio %.3g)"
        % (what, float((err / lim).max()) if err.size else 0.0, k, n_plain, err.size,
           float((err / plain).max()) if err.size else 0.0))
    bad = err > lim
    if bad.any():
        i = np.argwhere(bad)[0]
        raise AssertionError("%s: %d/%d elements out of tolerance; first at %s: got %r want %r absum %r"
                             % (what, int(bad.sum()), bad.size, tuple(i), got[tuple(i)], want[tuple(i)],
                                absum[tuple(i)]))


def trees_np(trees_t: torch.Tensor) -> np.ndarray:
    return trees_t.cpu().numpy().view(np.uint32).reshape(-1, 4)


def log(msg):
    print(msg, flush=True)


@functools.lru_cache(maxsize=None)
def workload_occupancy(key: str):
    wl = synth.WORKLOADS[key]
    if wl.dense_features:
        if key == "c1":
            occ = synth.occupancy(wl)
            dense = occ[..., None].astype(np.float32)
            return occ, dense
        return synth.facade_input(wl)
    return synth.occupancy(wl), None


def sample_rows(n_leaves: int, info: np.ndarray, k: int, seed: int) -> np.ndarray:
    """Random rows plus rows of every leaf size present, and the first/last rows."""
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(n_leaves, size=min(k, n_leaves), replace=False).tolist())
    bits = (info & np.uint64(1023)).astype(np.int64)
    for lo, hi in ((0, 1), (1, 9), (9, 73), (73, 585)):
        idx = np.nonzero((bits >= lo) & (bits < hi))[0]
        if idx.size:
            rows.update(rng.choice(idx, size=min(64, idx.size), replace=False).tolist())
    rows.update([0, n_leaves - 1])
    return np.array(sorted(rows), dtype=np.int64)
