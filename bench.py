"""Benchmark of the grid-octree hot path on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--config c4] [--no-cpu-baseline]

A step is one pass of the whole hot path over one batch of the workload:
octree build from the resident occupancy grid (with leaf counts and prefix
scan), input features, and the layer stack (conv3x3x3 with fused ReLU,
max-pooling, unpooling).  Inputs are resident in HBM before timing starts.

Prints one JSON line.  `value` is leaf-cells per second of whole steps
(leaves of the convolution's input octree x steps / wall time of the steps);
the convolution alone is reported as conv_leaf_cells_per_s and
dense_voxels_per_s, and its roofline fraction (fp32 MFMA peak) in
`roofline`, timed with HIP events on the stream the kernel runs on.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_TFLOPS = 157.3   # MI355X dense fp32 (vector and MFMA)
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="c4", choices=["c1", "c2", "c3", "c4", "c5", "unet"])
    ap.add_argument("--impl", default="auto", choices=["auto", "generic", "mfma"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--report", choices=["memory", "truncated"], default=None,
                    help="print a report table instead of the bench line")
    ap.add_argument("--bwd-steps", type=int, default=3,
                    help="backward passes timed after the forward steps (0: none)")
    ap.add_argument("--cpu-rows", type=int, default=500000,
                    help="leaves in the oracle's timed sample")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="host threads of the oracle's timed run (0: all)")
    ap.add_argument("--print-hash", action="store_true",
                    help="print the conv translation unit's source hash and exit")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device to device three times (a plain copy of "
                         "known size, to calibrate rocprofv3 FETCH_SIZE / WRITE_SIZE) and exit")
    return ap.parse_args()


def copy_probe(mib):
    import torch
    torch.cuda.set_device(0)
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": 4 * n, "copies": 3}), flush=True)


def measured_traffic(config):
    """HBM bytes per conv call from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary (copy-calibrated), or None when the summary is for
    another workload or the convolution source has changed since."""
    if config != "c4":
        return None
    path = os.path.join(ROOT, "profiles", "traffic_conv_surf256_b16.md")
    try:
        text = open(path).read()
        h = conv_source_hash()
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines() if ": " in line and
                  line.split(": ", 1)[0] in ("conv_source_sha256_16", "traffic_bytes_per_conv"))
    if fields.get("conv_source_sha256_16") != h:
        return None
    return float(fields["traffic_bytes_per_conv"])


# Every file of the convolution's translation unit: a change to any of them
# can change the kernels the traffic counters were taken on.
CONV_TU = ("oc_conv.hip", "oc_conv_gemm.inc", "oc_conv_bwd.inc", "oc_internal.h", "oc_device.h")


def conv_source_hash():
    """sha256 (first 16 hex digits) over the conv translation unit's files."""
    import hashlib
    h = hashlib.sha256()
    for name in CONV_TU:
        h.update(name.encode())
        h.update(open(os.path.join(ROOT, "paper_1611_05009_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:16]


def conv_flops_bytes(n_leaves, n_trees, cin, cout):
    """Algorithmic work of one conv layer: one (27 cin) x cout contraction per
    leaf; every input and output row read/written once, plus bit strings,
    prefix and weights."""
    flops = 2.0 * 27 * cin * cout * n_leaves
    nbytes = 4.0 * n_leaves * (cin + cout) + 24.0 * n_trees + 4.0 * (27 * cin * cout + cout)
    return flops, nbytes


def per_op_rooflines(W, recs, conv_ms, prep_ms, op_ms):
    """Per op of one step: time, leaf-cells/s, dense voxels/s and the
    fraction of the roofline that binds it (conv: max of the fp32 MFMA time
    and the HBM time of its algorithmic work; build, pool, unpool: HBM bytes
    of rows, bit strings and prefixes read and written)."""
    rows = []
    k = 0
    per_name = {}
    for r in recs:
        if r.op in ("input", "save"):
            if r.op == "input":
                nb = W.dense_voxels + 24.0 * r.g_out.n_trees
                per_name.setdefault("build", []).append(nb)
            continue
        if r.op == "conv":
            p = r.params
            t = conv_ms[k] * 1e-3
            fl, nb = conv_flops_bytes(r.g_in.n_leaves, r.g_in.n_trees, p["cin"], p["cout"])
            t_roof = max(fl / (PEAK_FP32_TFLOPS * 1e12), nb / (PEAK_HBM_GBS * 1e9))
            rows.append({"op": "conv%dx%d" % (p["cin"], p["cout"]), "ms": conv_ms[k],
                         "prepare_ms": prep_ms[k], "leaves": r.g_in.n_leaves,
                         "leaf_cells_per_s": r.g_in.n_leaves / t,
                         "dense_voxels_per_s": 512.0 * r.g_in.n_trees / t,
                         "bound": "mfma" if fl / (PEAK_FP32_TFLOPS * 1e12) >= nb / (PEAK_HBM_GBS * 1e9) else "hbm",
                         "frac": t_roof / t, "frac_with_prepare": t_roof / (t + prep_ms[k] * 1e-3)})
            k += 1
            continue
        c = r.x_in.shape[1]
        nb = 4.0 * c * (r.g_in.n_leaves + r.g_out.n_leaves) + 24.0 * (r.g_in.n_trees + r.g_out.n_trees)
        per_name.setdefault(r.op, []).append(nb)
    for name, nbs in per_name.items():
        ms = op_ms.get(name)
        if not ms:
            continue
        nb = sum(nbs)
        rows.append({"op": name, "calls": len(nbs), "ms": ms, "alg_bytes": nb, "bound": "hbm",
                     "frac": nb / (PEAK_HBM_GBS * 1e9) / (ms * 1e-3),
                     "note": "structure call included (it synchronizes to return the leaf count)"
                     if name != "concat" else ""})
    return rows


def cpu_baseline(W, rows_wanted, threads=0):
    """The oracle (never tuned) on a random sample of the workload's leaves,
    for the first conv layer: leaf-cells per second on the host cores
    (threads > 0: on that many)."""
    sys.path.insert(0, os.path.join(ROOT, "oracle"))
    import octref as O
    if threads > 0:
        O.set_num_threads(threads)
    import torch
    from paper_1611_05009_amd import pipeline

    recs = []
    pipeline.run_step(W, recs)
    torch.cuda.synchronize()
    conv = next(r for r in recs if r.op == "conv")
    g = conv.g_in
    ref = O.make_grid(g.trees.cpu().numpy().view(np.uint32).reshape(-1, 4), *g.dims())
    x = conv.x_in.cpu().numpy()
    info = O.leaf_info(ref)
    rng = np.random.default_rng(7)
    rows = np.sort(rng.choice(ref.n_leaves, size=min(rows_wanted, ref.n_leaves), replace=False))
    w = conv.params["w"].cpu().numpy()
    b = conv.params["b"].cpu().numpy()
    t0 = time.perf_counter()
    O.conv3_sampled(ref, x, w, b, conv.params["relu"], rows, info=info)
    dt = time.perf_counter() - t0
    return {
        "value": rows.size / dt,
        "unit": "leaf-cells/s",
        "cores": O.num_threads(),
        "kind": "oracle",
        "sample": "conv layer 0 on %d uniformly drawn leaves of %d (%.1f s, fp64, rowmaps built per sample)"
                  % (rows.size, ref.n_leaves, dt),
    }


def backward_times(W, steps):
    """Milliseconds per backward pass of the step's layers, by op (HIP events
    around each call), after one untimed warmup pass.  Outside the forward's
    timed region and not part of `value`."""
    import torch
    from paper_1611_05009_amd import pipeline

    recs = []
    g, x = pipeline.run_step(W, recs)
    gen = torch.Generator(device="cuda").manual_seed(7)
    dy = torch.randn(x.shape, generator=gen, device="cuda", dtype=torch.float32)
    pipeline.run_backward(W, recs, dy)
    torch.cuda.synchronize()
    evs = []

    def op_timer(name):
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        evs.append((name, s, e))
        return s, e

    for _ in range(steps):
        pipeline.run_backward(W, recs, dy, op_timer=op_timer)
    torch.cuda.synchronize()
    ms = {}
    for name, s, e in evs:
        ms[name] = ms.get(name, 0.0) + s.elapsed_time(e) / steps
    print("backward timed: %s" % ms, file=sys.stderr, flush=True)
    return ms


def memory_report():
    """Grid-octree vs dense bytes (1 and 8 features) of synthetic surface
    shapes at 8^3 .. 256^3, structures built on the GPU."""
    import torch
    from paper_1611_05009_amd import octnet as oc
    from paper_1611_05009_amd import reports as R
    from paper_1611_05009_amd import synth

    oc.lib()
    print("| grid | shape size (voxels) | occupancy % | leaves | dense MB (c=1) | octree MB (c=1) | dense MB (c=8) | octree MB (c=8) |")
    print("|---|---|---|---|---|---|---|---|")
    rng = np.random.default_rng(2017)
    for res in (8, 16, 32, 64, 128, 256):
        for frac in (0.3, 0.6, 0.95):
            size = max(2.0, frac * res)
            occ = synth.surface_sample(rng, res, size * 0.9, size)
            g = oc.build(torch.from_numpy(occ[None]).cuda())
            n_trees = (res // 8) ** 3
            vox = res ** 3
            print("| %d^3 | %.0f | %.2f | %d | %.3f | %.3f | %.3f | %.3f |" % (
                res, size, 100.0 * occ.mean(), g.n_leaves,
                R.dense_bytes(vox, 1) / 1e6, R.octree_bytes(n_trees, g.n_leaves, 1) / 1e6,
                R.dense_bytes(vox, 8) / 1e6, R.octree_bytes(n_trees, g.n_leaves, 8) / 1e6), flush=True)


def truncated_report(config):
    """Products per channel pair of the three schemes over the workload's
    first conv layer, and the measured time of the truncated kernel (the
    paper's scheme) beside the default path on that layer."""
    import torch
    from paper_1611_05009_amd import octnet as oc
    from paper_1611_05009_amd import pipeline
    from paper_1611_05009_amd import reports as R

    oc.lib()
    W = pipeline.Workload(config)
    recs = []
    pipeline.run_step(W, recs)
    conv = next(r for r in recs if r.op == "conv")
    g, x, p = conv.g_in, conv.x_in, conv.params
    info = oc.leaf_index(g).cpu().numpy()
    bits = info & 1023
    hist = {8: int((bits == 0).sum()), 4: int(((bits >= 1) & (bits < 9)).sum()),
            2: int(((bits >= 9) & (bits < 73)).sum()), 1: int((bits >= 73).sum())}
    prods = R.workload_products(hist, p["cin"], p["cout"])
    times = {}
    for impl in ("auto", "truncated"):
        oc.conv3x3x3(g, x, p["w"], p["b"], impl=impl)
        torch.cuda.synchronize()
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        s.record()
        oc.conv3x3x3(g, x, p["w"], p["b"], impl=impl)
        e.record()
        torch.cuda.synchronize()
        times[impl] = s.elapsed_time(e)
    print("| workload | conv | leaves (edge 8/4/2/1) | naive products | truncated products | window-sum products | truncated kernel ms | default path ms |")
    print("|---|---|---|---|---|---|---|---|")
    print("| %s | %dx%d | %d / %d / %d / %d | %.4g | %.4g | %.4g | %.2f | %.2f |" % (
        config, p["cin"], p["cout"], hist[8], hist[4], hist[2], hist[1], prods["naive"],
        prods["truncated"], prods["window_sums"], times["truncated"], times["auto"]))


def main():
    args = parse()
    if args.report == "memory":
        memory_report()
        return
    if args.report == "truncated":
        truncated_report(args.config)
        return
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.print_hash:
        print(conv_source_hash())
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(see DESIGN.md for how the work would shard)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_1611_05009_amd import octnet as oc
    from paper_1611_05009_amd import pipeline

    oc.lib()
    torch.cuda.set_device(0)
    t_gen = time.perf_counter()
    W = pipeline.Workload(args.config)
    t_gen = time.perf_counter() - t_gen
    print("inputs ready (%.1f s): %s, %d leaves" % (t_gen, args.config, W.n_leaves), file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    events = []
    prep_events = []

    def timer():
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        events.append((s, e))
        return s, e

    def prep_timer():
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        prep_events.append((s, e))
        return s, e

    op_events = []

    def op_timer(name):
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        op_events.append((name, s, e))
        return s, e

    for _ in range(args.warmup):
        pipeline.run_step(W, impl=args.impl)
    torch.cuda.synchronize()
    print("warmup done", file=sys.stderr, flush=True)

    events.clear()
    prep_events.clear()
    op_events.clear()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        pipeline.run_step(W, conv_timer=timer, impl=args.impl, prep_timer=prep_timer,
                          op_timer=op_timer)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_step = 1e3 * dt / args.steps

    convs = [L for L in W.layers if L[0] == "conv"]
    n_conv = len(convs)
    per_layer_ms = [0.0] * n_conv
    for k, (s, e) in enumerate(events):
        per_layer_ms[k % n_conv] += s.elapsed_time(e) / args.steps
    prep_ms = [0.0] * n_conv
    for k, (s, e) in enumerate(prep_events):
        prep_ms[k % n_conv] += s.elapsed_time(e) / args.steps
    # Build, pool and unpool, each summed over its calls in a step (the
    # structure calls synchronize to return leaf counts to the host).
    op_ms = {}
    for name, s, e in op_events:
        op_ms[name] = op_ms.get(name, 0.0) + s.elapsed_time(e) / args.steps
    # Dominant kernel: the conv layer with the longest execute (the only one
    # in the 256^3 workload); its leaf count from one recorded pass.
    recs = []
    pipeline.run_step(W, recs)
    conv_recs = [r for r in recs if r.op == "conv"]
    kd = max(range(n_conv), key=lambda k: per_layer_ms[k])
    p0 = convs[kd][1]
    g0 = conv_recs[kd].g_in
    n_trees = g0.n_trees
    flops, nbytes = conv_flops_bytes(g0.n_leaves, n_trees, p0["cin"], p0["cout"])
    t_conv = per_layer_ms[kd] * 1e-3
    achieved = flops / t_conv / 1e12
    out = {
        "metric": "octree conv3x3x3 leaf-cells/s + effective dense voxels/s at 256^3; % roofline",
        "value": W.n_leaves * args.steps / dt,
        "unit": "leaf-cells/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": W.wl.description,
            "key": args.config,
            "batch": W.batch,
            "grid": list(W.occ.shape[1:]),
            "n_leaves": W.n_leaves,
            "n_trees": n_trees,
            "layers": [L.op if L.op != "conv" else "conv%dx%d" % (L.cin, L.cout) for L in W.wl.layers],
            "impl": args.impl,
        },
        "conv_ms": per_layer_ms,
        "conv_prepare_ms": prep_ms,
        "op_ms": op_ms,
        "conv_leaf_cells_per_s": g0.n_leaves / t_conv,
        "dense_voxels_per_s": 512.0 * n_trees / t_conv,
        "roofline": {
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_FP32_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_FP32_TFLOPS,
            "traffic": measured_traffic(args.config),
            "kernel": "conv3x3x3 execute, layer %d (%dx%d, %d leaves): one HIP-event pair around all its launches (for a fused MFMA variant: the unit-voxel kernel, the boundary sums and the four cell kernels; otherwise window sums of row chunks and the MFMA GEMM); prepare, which depends on the structure and weights only, is timed apart as conv_prepare_ms and is part of every step" % (kd, p0["cin"], p0["cout"], g0.n_leaves),
            "alg_flops": flops,
            "alg_bytes": nbytes,
            "hbm_frac": nbytes / t_conv / 1e9 / PEAK_HBM_GBS,
            # The prepare call (structure and weight tables) runs once per
            # conv in every step: the fraction with it counted.
            "frac_with_prepare": flops / (t_conv + prep_ms[kd] * 1e-3) / 1e12 / PEAK_FP32_TFLOPS,
            "prepare_ms": prep_ms[kd],
        },
        "per_op": per_op_rooflines(W, recs, per_layer_ms, prep_ms, op_ms),
    }
    if args.bwd_steps > 0:
        bms = backward_times(W, args.bwd_steps)
        out["backward_ms"] = bms
        # Matrix-core rates of the conv gradients over all conv layers: each
        # gradient is 2 * 27 * Cin * Cout flops per leaf, like the forward.
        fl = sum(2.0 * 27 * r.params["cin"] * r.params["cout"] * r.g_in.n_leaves for r in conv_recs)
        rates = {}
        for name in ("conv_bwd_input", "conv_bwd_weight"):
            if bms.get(name):
                tf = fl / (bms[name] * 1e-3) / 1e12
                rates[name] = {"achieved_tflops": tf, "frac_of_fp32_mfma_peak": tf / PEAK_FP32_TFLOPS}
        out["backward_roofline"] = rates
    if not args.no_cpu_baseline:
        print("timing the oracle on the host", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(W, args.cpu_rows, args.cpu_threads)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
