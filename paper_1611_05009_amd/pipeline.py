"""One pass of the grid-octree hot path over a workload's batch.

A step builds the octree from the resident occupancy grid, forms the input
leaf features (ten2oc of a dense input, or resident per-leaf features), and
runs the layer stack (conv3x3x3 with fused bias/ReLU, 2x2x2 max-pooling,
plain or guided 2x2x2 unpooling).  Every op is a call into the HIP library.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

from . import octnet as oc
from . import synth


@dataclass
class OpRecord:
    op: str
    g_in: oc.Octree
    x_in: torch.Tensor
    g_out: oc.Octree
    x_out: torch.Tensor
    params: dict = field(default_factory=dict)


class Workload:
    """Inputs of one workload, resident on the GPU, and its layer stack."""

    def __init__(self, key: str, batch: int | None = None, device: str = "cuda"):
        self.key = key
        self.wl = synth.WORKLOADS[key]
        self.batch = self.wl.batch if batch is None else batch
        self.device = torch.device(device)
        wl = self.wl
        self.points = None
        if wl.points:
            pts, bidx, feat, labels = synth.point_cloud(wl, batch=self.batch)
            self.points = (torch.from_numpy(pts).to(self.device), torch.from_numpy(bidx).to(self.device),
                           torch.from_numpy(feat).to(self.device), torch.from_numpy(labels).to(self.device))
            self.points_np = (pts, bidx, feat, labels)
            occ = None  # voxelised on the GPU by every step
            self.dense = None
        elif wl.dense_features:
            if key == "c1":
                occ = synth.occupancy(wl, batch=self.batch)
                dense = occ[..., None].astype(np.float32)
            else:
                occ, dense = synth.facade_input(wl, batch=self.batch)
            self.dense = torch.from_numpy(dense).to(self.device)
        else:
            occ = synth.occupancy(wl, batch=self.batch)
            self.dense = None
        self.occ_np = occ
        if occ is None:
            self.occ = oc.points_voxelize(self.points[0], self.batch, wl.grid, wl.grid, wl.grid,
                                          batch=self.points[1])
        else:
            self.occ = torch.from_numpy(occ).to(self.device)
        g = oc.build(self.occ)
        self.n_leaves = g.n_leaves
        self.features = None
        if not wl.dense_features and not wl.points:
            self.features = torch.from_numpy(synth.leaf_features(wl, g.n_leaves, wl.cin)).to(self.device)
        # Conv layers with their fused ReLU flags.
        self.layers = []
        k = 0
        ops = wl.layers
        for i, L in enumerate(ops):
            if L.op == "relu":
                continue
            if L.op == "conv":
                w, b = synth.conv_weights(wl, k, L.cin, L.cout)
                relu = i + 1 < len(ops) and ops[i + 1].op == "relu"
                self.layers.append(("conv", dict(w=torch.from_numpy(w).to(self.device),
                                                 b=torch.from_numpy(b).to(self.device),
                                                 cin=L.cin, cout=L.cout, relu=relu, index=k)))
                k += 1
            else:
                self.layers.append((L.op, {}))

    @property
    def dense_voxels(self) -> int:
        return int(np.prod(self.occ.shape))


def run_step(W: Workload, records: list | None = None, conv_timer=None, impl: str = "auto",
             prep_timer=None, op_timer=None):
    """One pass of the hot path.  Returns (structure, features) at the end.
    conv_timer() returns a (start, end) event pair that brackets each
    convolution proper (execute); prep_timer() one that brackets each
    convolution's prepare (structure- and weight-dependent tables);
    op_timer(name) one that brackets the build ("build") and each pool or
    unpool ("pool", "unpool", "unpool_guided")."""
    def timed(name, fn):
        if op_timer is None:
            return fn()
        s, e = op_timer(name)
        s.record()
        r = fn()
        e.record()
        return r

    if W.points is not None:
        # Point cloud: voxelise, build, then the per-leaf occupancy flag and
        # mean point features.
        pts, bidx, feat, _ = W.points
        n, gdim = W.batch, W.wl.grid

        def from_points():
            occ = oc.points_voxelize(pts, n, gdim, gdim, gdim, batch=bidx)
            gg = oc.build(occ)
            rows = oc.points_leaf_rows(gg, pts, bidx)
            return gg, oc.points_average(gg, rows, feat)

        g, x = timed("build", from_points)
    else:
        g = timed("build", lambda: oc.build(W.occ))
        x = oc.ten2oc(g, W.dense, "avg") if W.dense is not None else W.features
    if records is not None:
        records.append(OpRecord("input", g, x, g, x))
    guides = []
    skips = []
    for op, p in W.layers:
        g_in, x_in = g, x
        if op == "save":
            skips.append(x)
        elif op == "concat":
            x = timed("concat", lambda: oc.concat(skips.pop(), x_in))
        elif op == "conv":
            if prep_timer is not None:
                ps, pe = prep_timer()
                ps.record()
            ws = oc.conv3x3x3_prepare(g, p["w"])
            if prep_timer is not None:
                pe.record()
            if conv_timer is not None:
                s, e = conv_timer()
                s.record()
            x = oc.conv3x3x3_execute(g, x, p["cout"], ws, p["b"], relu=p["relu"], impl=impl)
            if conv_timer is not None:
                e.record()
        elif op == "pool":
            guides.append(g)
            g, x = timed("pool", lambda: oc.pool2(g_in, x_in))
        elif op == "unpool":
            g, x = timed("unpool", lambda: oc.unpool2(g_in, x_in))
        elif op == "unpool_guided":
            guide = guides.pop()
            g, x = timed("unpool_guided", lambda: oc.unpool2(g_in, x_in, guide=guide))
        else:
            raise ValueError(op)
        if records is not None:
            records.append(OpRecord(op, g_in, x_in, g, x, p))
    return g, x


def run_backward(W: Workload, records: list, dy: torch.Tensor, op_timer=None, trace: list | None = None):
    """Gradients of one pass, from dy (the gradient of the last output)
    back through the layer stack recorded by run_step(W, records).  Returns
    (gradient of the input leaf features, {conv index: (dweight, dbias)}).
    op_timer(name), as in run_step, brackets each call: "unpool_bwd",
    "pool_bwd", "relu_bwd", "conv_bwd_input", "conv_bwd_weight" (the
    weight and bias gradients), "concat_bwd" and "add" (skip connections).  trace, when given, receives (record,
    gradient in, gradients out) for each op: out is the input gradient, or
    (relu-masked gradient, input gradient, dweight, dbias) for a conv."""
    def timed(name, fn):
        if op_timer is None:
            return fn()
        s, e = op_timer(name)
        s.record()
        r = fn()
        e.record()
        return r

    grads = {}
    skip_grads = []
    for rec in reversed(records):
        if rec.op == "input":
            break
        dy_in = dy
        if rec.op == "concat":
            # The concat took [saved encoder output, decoder features].
            ca = rec.x_out.shape[1] - rec.x_in.shape[1]
            d_enc, dy = timed("concat_bwd", lambda: oc.concat_backward(dy_in, ca))
            skip_grads.append(d_enc)
            out = (d_enc, dy)
        elif rec.op == "save":
            # The saved output also fed the concat: its gradients add up.
            dy = timed("add", lambda: oc.add(dy_in, skip_grads.pop()))
            out = dy
        elif rec.op in ("unpool", "unpool_guided"):
            dy = timed("unpool_bwd", lambda: oc.unpool2_backward(rec.g_in, rec.g_out, dy))
            out = dy
        elif rec.op == "pool":
            dy = timed("pool_bwd", lambda: oc.pool2_max_backward(rec.g_in, rec.x_in, rec.g_out, dy))
            out = dy
        elif rec.op == "conv":
            p = rec.params
            if p["relu"]:
                dy = timed("relu_bwd", lambda: oc.relu_backward(rec.x_out, dy))
            dyc = dy
            _, dw, db = timed("conv_bwd_weight", lambda: oc.conv3x3x3_backward(
                rec.g_in, rec.x_in, p["w"], dyc, need_input=False))
            grads[p["index"]] = (dw, db)
            dy = timed("conv_bwd_input", lambda: oc.conv3x3x3_backward(
                rec.g_in, None, p["w"], dyc, need_weight=False, need_bias=False)[0])
            out = (dyc, dy, dw, db)
        else:
            raise ValueError(rec.op)
        if trace is not None:
            trace.append((rec, dy_in, out))
    return dy, grads
