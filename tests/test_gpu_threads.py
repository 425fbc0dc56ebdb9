"""The library is stateless and thread-safe: per-device limits are queried
once per device under std::call_once, the kernels' constant tables are
initialised at load time, and every call works only on the buffers it is
given.  These tests call it from several host threads at once, each on its
own stream with its own workspace, and compare every result bit for bit with
a sequential run (the kernels are deterministic)."""
import os
import subprocess
import sys
import threading

import numpy as np
import pytest
import torch

from common import log

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


# Run in a fresh process, so that the library's very first calls (the
# per-device queries included) come from 8 threads at once.
_COLD_START = r"""
import sys, threading
import numpy as np, torch
sys.path.insert(0, %(root)r)
from paper_1611_05009_amd import octnet as oc, synth
torch.cuda.set_device(0)
rng = np.random.default_rng(5)
words = synth.random_trees(rng, 2, 3, 4, 3, 0.7, 0.5, 0.5)
g = oc.from_trees(torch.from_numpy(words.view(np.int32)).cuda(), 2, 3, 4, 3)
x = torch.from_numpy(rng.standard_normal((g.n_leaves, 32)).astype(np.float32)).cuda()
w = torch.from_numpy((rng.standard_normal((32, 32, 3, 3, 3)) / 30).astype(np.float32)).cuda()
torch.cuda.synchronize()
res = [None] * 8
go = threading.Barrier(8)
def work(k):
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        go.wait()
        y = oc.conv3x3x3(g, x, w, impl="mfma")
        dx, dw, db = oc.conv3x3x3_backward(g, x, w, y)
    s.synchronize()
    res[k] = [t.cpu() for t in (y, dx, dw, db)]
ts = [threading.Thread(target=work, args=(k,)) for k in range(8)]
for t in ts: t.start()
for t in ts: t.join()
y = oc.conv3x3x3(g, x, w, impl="mfma")
ref = [t.cpu() for t in (y,) + oc.conv3x3x3_backward(g, x, w, y)]
bad = [k for k in range(8) if res[k] is None or not all(torch.equal(a, b) for a, b in zip(res[k], ref))]
print("cold-start threads: %%d leaves, mismatching threads %%s" %% (g.n_leaves, bad), flush=True)
sys.exit(1 if bad else 0)
"""


def test_first_calls_from_eight_threads():
    log("cold start in a child process")
    r = subprocess.run([sys.executable, "-c", _COLD_START % {"root": ROOT}], capture_output=True,
                       text=True, timeout=300)
    log(r.stdout.strip())
    assert r.returncode == 0, r.stdout + r.stderr[-2000:]


def test_concurrent_calls_match_sequential():
    from paper_1611_05009_amd import octnet as oc
    from paper_1611_05009_amd import synth
    oc.lib()
    rng = np.random.default_rng(8)
    words = synth.random_trees(rng, 2, 4, 3, 3, 0.8, 0.5, 0.5)
    g = oc.from_trees(torch.from_numpy(words.view(np.int32)).cuda(), 2, 4, 3, 3)
    cases = [(32, 32), (16, 32), (8, 16), (4, 16), (32, 8), (64, 64)]
    xs = {c: torch.from_numpy(rng.standard_normal((g.n_leaves, c[0])).astype(np.float32)).cuda() for c in cases}
    ws = {c: torch.from_numpy((rng.standard_normal((c[1], c[0], 3, 3, 3)) / 20).astype(np.float32)).cuda()
          for c in cases}
    ref = {c: oc.conv3x3x3(g, xs[c], ws[c], impl="auto").cpu() for c in cases}
    torch.cuda.synchronize()
    out = {}
    errs = []

    def work(c):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                ys = [oc.conv3x3x3(g, xs[c], ws[c], impl="auto") for _ in range(4)]
            s.synchronize()
            out[c] = [y.cpu() for y in ys]
        except Exception as e:  # reported below
            errs.append((c, repr(e)))

    ts = [threading.Thread(target=work, args=(c,)) for c in cases]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert not errs, errs
    for c in cases:
        for y in out[c]:
            assert torch.equal(y, ref[c]), c
