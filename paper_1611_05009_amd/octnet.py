"""Python binding of the grid-octree HIP library (liboctnet_hip.so).

Argument marshalling only: every step runs in the library's HIP kernels.
PyTorch supplies device memory and the current HIP stream.  There is no
fallback path: if the library is missing, every call raises.

Tensors: trees int32 [n_trees, 4] (the uint32 bit words), prefix int64
[n_trees + 1], leaf data float32 [n_leaves, C], all on the GPU.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboctnet_hip.so")

OC_OK = 0
OC_SPLIT_MIXED, OC_SPLIT_ANY = 0, 1
OC_POOL_AVG, OC_POOL_MAX = 0, 1
OC_CONV_AUTO, OC_CONV_GENERIC, OC_CONV_MFMA, OC_CONV_GEMM, OC_CONV_TRUNCATED = 0, 1, 2, 3, 4

_IMPL = {"auto": OC_CONV_AUTO, "generic": OC_CONV_GENERIC, "mfma": OC_CONV_MFMA, "gemm": OC_CONV_GEMM,
         "truncated": OC_CONV_TRUNCATED}

_P = ctypes.c_void_p
_I = ctypes.c_int
_L = ctypes.c_int64
_S = ctypes.c_size_t

# name -> (restype, argtypes); mirrors include/octnet_hip.h
SIGNATURES = {
    "oc_error_string": (ctypes.c_char_p, [_I]),
    "oc_last_error": (ctypes.c_char_p, []),
    "oc_version": (_I, []),
    "oc_structure_workspace": (_S, [_L]),
    "oc_build": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _S, _P]),
    "oc_build_noalloc": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P]),
    "oc_prefix": (_I, [_P, _L, _P, _P, _P, _S, _P]),
    "oc_validate": (_I, [_P, _L, _P, _P, _S, _P]),
    "oc_leaf_index": (_I, [_P, _P, _L, _P, _P]),
    "oc_rowmap": (_I, [_P, _P, _I, _I, _I, _I, _P, _P]),
    "oc_oc2ten": (_I, [_P, _P, _I, _I, _I, _I, _P, _I, _P, _P]),
    "oc_ten2oc": (_I, [_P, _P, _I, _I, _I, _I, _P, _I, _I, _P, _P]),
    "oc_conv3x3x3_workspace": (_I, [_L, _L, _I, _I, _P]),
    "oc_conv3x3x3_workspace_exact": (_I, [_P, _I, _I, _I, _I, _L, _I, _I, _P, _P, _P]),
    "oc_conv3x3x3_workspace_slots": (_I, [_L, _L, _I, _I, _L, _P]),
    "oc_conv3x3x3_workspace_capacity": (_I, [_L, _L, _I, _I, ctypes.c_size_t, _P]),
    "oc_conv3x3x3": (_I, [_P, _P, _I, _I, _I, _I, _L, _P, _I, _P, _P, _I, _I, _P, _P, _S, _P]),
    "oc_conv3x3x3_ex": (_I, [_P, _P, _I, _I, _I, _I, _L, _P, _I, _P, _P, _I, _I, _P, _P, _S, _I, _P]),
    "oc_conv3x3x3_prepare": (_I, [_P, _P, _I, _I, _I, _I, _L, _P, _I, _I, _P, _S, _P]),
    "oc_conv3x3x3_execute": (_I, [_P, _P, _I, _I, _I, _I, _L, _P, _I, _P, _I, _I, _P, _P, _S, _I, _P]),
    "oc_conv3x3x3_mfma_supported": (_I, [_I, _I]),
    "oc_pool2_structure": (_I, [_P, _I, _I, _I, _I, _P, _P, _P, _P, _S, _P]),
    "oc_pool2_max": (_I, [_P, _P, _I, _I, _I, _I, _P, _I, _P, _P, _P, _P]),
    "oc_unpool2_structure": (_I, [_P, _I, _I, _I, _I, _P, _P, _P, _P, _P, _S, _P]),
    "oc_unpool2": (_I, [_P, _P, _I, _I, _I, _I, _P, _I, _P, _P, _P, _P]),
    "oc_relu": (_I, [_P, _L, _P]),
    "oc_conv3x3x3_backward_workspace": (_I, [_L, _L, _I, _I, _P]),
    "oc_conv3x3x3_backward": (_I, [_P, _P, _I, _I, _I, _I, _L, _P, _I, _P, _I, _P, _P, _P, _P, _P,
                                   _S, _P]),
    "oc_pool2_max_backward": (_I, [_P, _P, _I, _I, _I, _I, _P, _I, _P, _P, _P, _P, _P]),
    "oc_unpool2_backward": (_I, [_P, _P, _I, _I, _I, _I, _L, _I, _P, _P, _P, _P, _P]),
    "oc_relu_backward": (_I, [_P, _P, _P, _L, _P]),
    "oc_concat": (_I, [_P, _I, _P, _I, _L, _P, _P]),
    "oc_concat_backward": (_I, [_P, _I, _I, _L, _P, _P, _P]),
    "oc_add": (_I, [_P, _P, _P, _L, _P]),
    "oc_points_voxelize": (_I, [_P, _P, _L, _I, _I, _I, _I, _P, _P]),
    "oc_points_leaf_rows": (_I, [_P, _P, _I, _I, _I, _I, _P, _P, _L, _P, _P]),
    "oc_points_workspace": (_S, [_L, _I]),
    "oc_points_average": (_I, [_P, _L, _P, _I, _L, _P, _P, _S, _P]),
    "oc_points_vote": (_I, [_P, _L, _P, _I, _L, _P, _P, _S, _P]),
}

_lib = None


class OctNetError(RuntimeError):
    pass


def lib():
    """Load liboctnet_hip.so; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise OctNetError(
                "liboctnet_hip.so is missing; build it with __graft_entry__.build() "
                "(hipcc --offload-arch=gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(rc: int, what: str) -> None:
    if rc != OC_OK:
        L = lib()
        raise OctNetError("%s failed: %s (%d): %s" % (
            what, L.oc_error_string(rc).decode(), rc, L.oc_last_error().decode()))


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise OctNetError("expected a GPU tensor")
    if not t.is_contiguous():
        raise OctNetError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev():
    return torch.device("cuda", torch.cuda.current_device())


@dataclass
class Octree:
    """Structure of a batch of hybrid grid-octrees (no features)."""

    n: int
    gd: int
    gh: int
    gw: int
    trees: torch.Tensor   # int32 [n_trees, 4]
    prefix: torch.Tensor  # int64 [n_trees + 1]
    n_leaves: int

    @property
    def n_trees(self) -> int:
        return self.n * self.gd * self.gh * self.gw

    @property
    def dense_shape(self):
        return (self.n, 8 * self.gd, 8 * self.gh, 8 * self.gw)

    def dims(self):
        return self.n, self.gd, self.gh, self.gw


def structure_workspace(n_trees: int) -> torch.Tensor:
    nbytes = lib().oc_structure_workspace(int(n_trees))
    return torch.empty(nbytes, dtype=torch.uint8, device=_dev())


def build(occ: torch.Tensor, rule: str = "mixed") -> Octree:
    """Octree from a uint8 occupancy tensor [N, 8gd, 8gh, 8gw] on the GPU."""
    if occ.dtype != torch.uint8 or occ.dim() != 4:
        raise OctNetError("occupancy must be uint8 [N, D, H, W]")
    n, D, H, W = occ.shape
    if D % 8 or H % 8 or W % 8:
        raise OctNetError("voxel grid dims must be multiples of 8")
    gd, gh, gw = D // 8, H // 8, W // 8
    nt = n * gd * gh * gw
    trees = torch.empty((nt, 4), dtype=torch.int32, device=occ.device)
    prefix = torch.empty(nt + 1, dtype=torch.int64, device=occ.device)
    ws = structure_workspace(nt)
    nl = ctypes.c_int64(0)
    _check(lib().oc_build(_ptr(occ), n, gd, gh, gw, OC_SPLIT_MIXED if rule == "mixed" else OC_SPLIT_ANY,
                          _ptr(trees), _ptr(prefix), ctypes.byref(nl), _ptr(ws), ws.numel(), _stream()),
           "oc_build")
    return Octree(n, gd, gh, gw, trees, prefix, nl.value)


def build_noalloc(occ: torch.Tensor, rule: str = "mixed", trees: torch.Tensor | None = None,
                  prefix: torch.Tensor | None = None) -> Octree:
    """build() through oc_build_noalloc: the library allocates nothing (its
    scratch is a static device array); trees and prefix may be passed in."""
    if occ.dtype != torch.uint8 or occ.dim() != 4:
        raise OctNetError("occupancy must be uint8 [N, D, H, W]")
    n, D, H, W = occ.shape
    if D % 8 or H % 8 or W % 8:
        raise OctNetError("voxel grid dims must be multiples of 8")
    gd, gh, gw = D // 8, H // 8, W // 8
    nt = n * gd * gh * gw
    if trees is None:
        trees = torch.empty((nt, 4), dtype=torch.int32, device=occ.device)
    if prefix is None:
        prefix = torch.empty(nt + 1, dtype=torch.int64, device=occ.device)
    if tuple(trees.shape) != (nt, 4) or tuple(prefix.shape) != (nt + 1,):
        raise OctNetError("trees must be [n_trees, 4] and prefix [n_trees + 1]")
    nl = ctypes.c_int64(0)
    _check(lib().oc_build_noalloc(_ptr(occ), n, gd, gh, gw, OC_SPLIT_MIXED if rule == "mixed" else OC_SPLIT_ANY,
                                  _ptr(trees), _ptr(prefix), ctypes.byref(nl), _stream()),
           "oc_build_noalloc")
    return Octree(n, gd, gh, gw, trees, prefix, nl.value)


def from_trees(trees: torch.Tensor, n: int, gd: int, gh: int, gw: int) -> Octree:
    """Octree from given bit words (prefix computed on the GPU)."""
    trees = trees.contiguous()
    nt = n * gd * gh * gw
    if tuple(trees.shape) != (nt, 4):
        raise OctNetError("trees must be [n_trees, 4]")
    prefix = torch.empty(nt + 1, dtype=torch.int64, device=trees.device)
    ws = structure_workspace(nt)
    nl = ctypes.c_int64(0)
    _check(lib().oc_prefix(_ptr(trees), nt, _ptr(prefix), ctypes.byref(nl), _ptr(ws), ws.numel(), _stream()),
           "oc_prefix")
    return Octree(n, gd, gh, gw, trees, prefix, nl.value)


def validate(g: Octree) -> int:
    """Number of non-canonical trees."""
    ws = structure_workspace(g.n_trees)
    bad = ctypes.c_int64(0)
    _check(lib().oc_validate(_ptr(g.trees), g.n_trees, ctypes.byref(bad), _ptr(ws), ws.numel(), _stream()),
           "oc_validate")
    return bad.value


def leaf_index(g: Octree) -> torch.Tensor:
    """int64 [n_leaves]: tree << 10 | bit index per row."""
    out = torch.empty(g.n_leaves, dtype=torch.int64, device=g.trees.device)
    _check(lib().oc_leaf_index(_ptr(g.trees), _ptr(g.prefix), g.n_trees, _ptr(out), _stream()),
           "oc_leaf_index")
    return out


def rowmap(g: Octree) -> torch.Tensor:
    out = torch.empty(g.dense_shape, dtype=torch.int64, device=g.trees.device)
    _check(lib().oc_rowmap(_ptr(g.trees), _ptr(g.prefix), *g.dims(), _ptr(out), _stream()), "oc_rowmap")
    return out


def oc2ten(g: Octree, data: torch.Tensor) -> torch.Tensor:
    c = data.shape[1]
    out = torch.empty(g.dense_shape + (c,), dtype=torch.float32, device=data.device)
    _check(lib().oc_oc2ten(_ptr(g.trees), _ptr(g.prefix), *g.dims(), _ptr(data), c, _ptr(out), _stream()),
           "oc_oc2ten")
    return out


def ten2oc(g: Octree, dense: torch.Tensor, pool: str = "avg") -> torch.Tensor:
    if tuple(dense.shape[:4]) != g.dense_shape:
        raise OctNetError("dense tensor shape does not match the grid")
    c = dense.shape[4]
    out = torch.empty((g.n_leaves, c), dtype=torch.float32, device=dense.device)
    _check(lib().oc_ten2oc(_ptr(g.trees), _ptr(g.prefix), *g.dims(), _ptr(dense), c,
                           OC_POOL_AVG if pool == "avg" else OC_POOL_MAX, _ptr(out), _stream()),
           "oc_ten2oc")
    return out


def conv_workspace_bytes(g: Octree, cin: int, cout: int, exact: bool = True) -> int:
    """Workspace of a convolution on g: sized for g's own boundary-sum slots
    (counted on the device, one synchronization) or, exact=False, the bound
    for every structure of g's size."""
    nb = ctypes.c_size_t(0)
    if exact:
        scratch = torch.empty(256, dtype=torch.uint8, device=g.trees.device)
        _check(lib().oc_conv3x3x3_workspace_exact(_ptr(g.trees), *g.dims(), g.n_leaves, cin, cout,
                                                  ctypes.byref(nb), _ptr(scratch), _stream()),
               "oc_conv3x3x3_workspace_exact")
    else:
        _check(lib().oc_conv3x3x3_workspace(g.n_trees, g.n_leaves, cin, cout, ctypes.byref(nb)),
               "oc_conv3x3x3_workspace")
    return nb.value


def mfma_supported(cin: int, cout: int) -> bool:
    return bool(lib().oc_conv3x3x3_mfma_supported(cin, cout))


def conv3x3x3(g: Octree, data: torch.Tensor, weight: torch.Tensor, bias: torch.Tensor | None = None,
              relu: bool = False, impl: str = "auto", ws: torch.Tensor | None = None,
              out: torch.Tensor | None = None) -> torch.Tensor:
    """Eq. 8 convolution; weight [Cout, Cin, 3, 3, 3] in Eq. 7's orientation."""
    cin = data.shape[1]
    cout = weight.shape[0]
    if tuple(weight.shape) != (cout, cin, 3, 3, 3):
        raise OctNetError("weight must be [Cout, Cin, 3, 3, 3]")
    if out is None:
        out = torch.empty((g.n_leaves, cout), dtype=torch.float32, device=data.device)
    if ws is None:
        ws = torch.empty(conv_workspace_bytes(g, cin, cout), dtype=torch.uint8, device=data.device)
    _check(lib().oc_conv3x3x3_ex(_ptr(g.trees), _ptr(g.prefix), *g.dims(), g.n_leaves, _ptr(data), cin,
                                 _ptr(weight), _ptr(bias), cout, int(bool(relu)), _ptr(out), _ptr(ws),
                                 ws.numel(), _IMPL[impl], _stream()),
           "oc_conv3x3x3")
    return out


def conv3x3x3_prepare(g: Octree, weight: torch.Tensor, ws: torch.Tensor | None = None) -> torch.Tensor:
    """Structure/weight preparation of the convolution; returns the workspace."""
    cout, cin = weight.shape[0], weight.shape[1]
    if ws is None:
        ws = torch.empty(conv_workspace_bytes(g, cin, cout), dtype=torch.uint8, device=weight.device)
    _check(lib().oc_conv3x3x3_prepare(_ptr(g.trees), _ptr(g.prefix), *g.dims(), g.n_leaves, _ptr(weight), cin,
                                      cout, _ptr(ws), ws.numel(), _stream()), "oc_conv3x3x3_prepare")
    return ws


def conv3x3x3_execute(g: Octree, data: torch.Tensor, cout: int, ws: torch.Tensor,
                      bias: torch.Tensor | None = None, relu: bool = False, impl: str = "auto",
                      out: torch.Tensor | None = None) -> torch.Tensor:
    """The convolution proper, from a workspace filled by conv3x3x3_prepare."""
    cin = data.shape[1]
    if out is None:
        out = torch.empty((g.n_leaves, cout), dtype=torch.float32, device=data.device)
    _check(lib().oc_conv3x3x3_execute(_ptr(g.trees), _ptr(g.prefix), *g.dims(), g.n_leaves, _ptr(data), cin,
                                      _ptr(bias), cout, int(bool(relu)), _ptr(out), _ptr(ws), ws.numel(),
                                      _IMPL[impl], _stream()), "oc_conv3x3x3_execute")
    return out


def pool2_structure(g: Octree) -> Octree:
    n, gd, gh, gw = g.dims()
    no = n * (gd // 2) * (gh // 2) * (gw // 2)
    trees = torch.empty((max(no, 1), 4), dtype=torch.int32, device=g.trees.device)
    prefix = torch.empty(no + 1, dtype=torch.int64, device=g.trees.device)
    ws = structure_workspace(no)
    nl = ctypes.c_int64(0)
    _check(lib().oc_pool2_structure(_ptr(g.trees), n, gd, gh, gw, _ptr(trees), _ptr(prefix), ctypes.byref(nl),
                                    _ptr(ws), ws.numel(), _stream()), "oc_pool2_structure")
    return Octree(n, gd // 2, gh // 2, gw // 2, trees, prefix, nl.value)


def pool2_max(g: Octree, data: torch.Tensor, out_g: Octree, out: torch.Tensor | None = None) -> torch.Tensor:
    c = data.shape[1]
    if out is None:
        out = torch.empty((out_g.n_leaves, c), dtype=torch.float32, device=data.device)
    _check(lib().oc_pool2_max(_ptr(g.trees), _ptr(g.prefix), *g.dims(), _ptr(data), c, _ptr(out_g.trees),
                              _ptr(out_g.prefix), _ptr(out), _stream()), "oc_pool2_max")
    return out


def pool2(g: Octree, data: torch.Tensor):
    og = pool2_structure(g)
    return og, pool2_max(g, data, og)


def unpool2_structure(g: Octree, guide: Octree | None = None) -> Octree:
    n, gd, gh, gw = g.dims()
    no = 8 * n * gd * gh * gw
    trees = torch.empty((no, 4), dtype=torch.int32, device=g.trees.device)
    prefix = torch.empty(no + 1, dtype=torch.int64, device=g.trees.device)
    ws = structure_workspace(no)
    nl = ctypes.c_int64(0)
    if guide is not None and guide.dims() != (n, 2 * gd, 2 * gh, 2 * gw):
        raise OctNetError("guide must have twice the input's tree grid")
    _check(lib().oc_unpool2_structure(_ptr(g.trees), n, gd, gh, gw, _ptr(guide.trees) if guide else None,
                                      _ptr(trees), _ptr(prefix), ctypes.byref(nl), _ptr(ws), ws.numel(),
                                      _stream()), "oc_unpool2_structure")
    return Octree(n, 2 * gd, 2 * gh, 2 * gw, trees, prefix, nl.value)


def unpool2_data(g: Octree, data: torch.Tensor, out_g: Octree, out: torch.Tensor | None = None) -> torch.Tensor:
    c = data.shape[1]
    if out is None:
        out = torch.empty((out_g.n_leaves, c), dtype=torch.float32, device=data.device)
    _check(lib().oc_unpool2(_ptr(g.trees), _ptr(g.prefix), *g.dims(), _ptr(data), c, _ptr(out_g.trees),
                            _ptr(out_g.prefix), _ptr(out), _stream()), "oc_unpool2")
    return out


def unpool2(g: Octree, data: torch.Tensor, guide: Octree | None = None):
    og = unpool2_structure(g, guide)
    return og, unpool2_data(g, data, og)


def relu_(data: torch.Tensor) -> torch.Tensor:
    _check(lib().oc_relu(_ptr(data), data.numel(), _stream()), "oc_relu")
    return data


def conv_backward_workspace_bytes(g: Octree, cin: int, cout: int) -> int:
    nb = ctypes.c_size_t(0)
    _check(lib().oc_conv3x3x3_backward_workspace(g.n_trees, g.n_leaves, cin, cout, ctypes.byref(nb)),
           "oc_conv3x3x3_backward_workspace")
    return nb.value


def conv3x3x3_backward(g: Octree, data: torch.Tensor | None, weight: torch.Tensor, dout: torch.Tensor,
                       need_input: bool = True, need_weight: bool = True, need_bias: bool = True,
                       ws: torch.Tensor | None = None):
    """Gradients of conv3x3x3 (without its ReLU) from dout [n_leaves, Cout]:
    (d input [n_leaves, Cin], d weight [Cout, Cin, 3, 3, 3], d bias [Cout]),
    None for each one not asked for."""
    cout, cin = weight.shape[0], weight.shape[1]
    if tuple(weight.shape) != (cout, cin, 3, 3, 3):
        raise OctNetError("weight must be [Cout, Cin, 3, 3, 3]")
    if tuple(dout.shape) != (g.n_leaves, cout):
        raise OctNetError("dout must be [n_leaves, Cout]")
    dev = dout.device
    din = torch.empty((g.n_leaves, cin), dtype=torch.float32, device=dev) if need_input else None
    dw = torch.empty((cout, cin, 3, 3, 3), dtype=torch.float32, device=dev) if need_weight else None
    db = torch.empty(cout, dtype=torch.float32, device=dev) if need_bias else None
    if need_weight and (data is None or tuple(data.shape) != (g.n_leaves, cin)):
        raise OctNetError("the weight gradient needs the input [n_leaves, Cin]")
    if ws is None:
        ws = torch.empty(conv_backward_workspace_bytes(g, cin, cout), dtype=torch.uint8, device=dev)
    _check(lib().oc_conv3x3x3_backward(_ptr(g.trees), _ptr(g.prefix), *g.dims(), g.n_leaves,
                                       _ptr(data) if need_weight else None, cin, _ptr(weight), cout,
                                       _ptr(dout), _ptr(din), _ptr(dw), _ptr(db), _ptr(ws), ws.numel(),
                                       _stream()), "oc_conv3x3x3_backward")
    return din, dw, db


def pool2_max_backward(g: Octree, data: torch.Tensor, out_g: Octree, dout: torch.Tensor) -> torch.Tensor:
    """Gradient of pool2_max with respect to its input leaves."""
    c = data.shape[1]
    if tuple(dout.shape) != (out_g.n_leaves, c):
        raise OctNetError("dout must be [out leaves, C]")
    din = torch.empty((g.n_leaves, c), dtype=torch.float32, device=data.device)
    _check(lib().oc_pool2_max_backward(_ptr(g.trees), _ptr(g.prefix), *g.dims(), _ptr(data), c,
                                       _ptr(out_g.trees), _ptr(out_g.prefix), _ptr(dout), _ptr(din),
                                       _stream()), "oc_pool2_max_backward")
    return din


def unpool2_backward(g: Octree, out_g: Octree, dout: torch.Tensor) -> torch.Tensor:
    """Gradient of unpool2_data (plain or guided) with respect to its input leaves."""
    c = dout.shape[1]
    if dout.shape[0] != out_g.n_leaves:
        raise OctNetError("dout must be [out leaves, C]")
    din = torch.empty((g.n_leaves, c), dtype=torch.float32, device=dout.device)
    _check(lib().oc_unpool2_backward(_ptr(g.trees), _ptr(g.prefix), *g.dims(), g.n_leaves, c,
                                     _ptr(out_g.trees), _ptr(out_g.prefix), _ptr(dout), _ptr(din),
                                     _stream()), "oc_unpool2_backward")
    return din


def relu_backward(out: torch.Tensor, dout: torch.Tensor, din: torch.Tensor | None = None) -> torch.Tensor:
    """dout where the ReLU output is positive, else 0 (din may be dout)."""
    if out.shape != dout.shape:
        raise OctNetError("out and dout must have one shape")
    if din is None:
        din = torch.empty_like(dout)
    _check(lib().oc_relu_backward(_ptr(out), _ptr(dout), _ptr(din), dout.numel(), _stream()),
           "oc_relu_backward")
    return din


def concat(a: torch.Tensor, b: torch.Tensor) -> torch.Tensor:
    """[a, b] along the channels of two leaf arrays on one structure."""
    if a.shape[0] != b.shape[0]:
        raise OctNetError("concat needs the same row count")
    out = torch.empty((a.shape[0], a.shape[1] + b.shape[1]), dtype=torch.float32, device=a.device)
    _check(lib().oc_concat(_ptr(a), a.shape[1], _ptr(b), b.shape[1], a.shape[0], _ptr(out), _stream()),
           "oc_concat")
    return out


def concat_backward(dout: torch.Tensor, ca: int):
    """Gradient of concat: (da [rows, ca], db [rows, C - ca])."""
    cb = dout.shape[1] - ca
    da = torch.empty((dout.shape[0], ca), dtype=torch.float32, device=dout.device)
    db = torch.empty((dout.shape[0], cb), dtype=torch.float32, device=dout.device)
    _check(lib().oc_concat_backward(_ptr(dout), ca, cb, dout.shape[0], _ptr(da), _ptr(db), _stream()),
           "oc_concat_backward")
    return da, db


def add(a: torch.Tensor, b: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
    """a + b (same shape); out may be a or b."""
    if a.shape != b.shape:
        raise OctNetError("add needs one shape")
    if out is None:
        out = torch.empty_like(a)
    _check(lib().oc_add(_ptr(a), _ptr(b), _ptr(out), a.numel(), _stream()), "oc_add")
    return out


def points_voxelize(pts: torch.Tensor, n: int, gd: int, gh: int, gw: int,
                    batch: torch.Tensor | None = None) -> torch.Tensor:
    """uint8 occupancy [n, 8gd, 8gh, 8gw] of a point cloud (pts [P, 3] in voxels)."""
    occ = torch.empty((n, 8 * gd, 8 * gh, 8 * gw), dtype=torch.uint8, device=pts.device)
    _check(lib().oc_points_voxelize(_ptr(pts), _ptr(batch), pts.shape[0], n, gd, gh, gw, _ptr(occ),
                                    _stream()), "oc_points_voxelize")
    return occ


def points_leaf_rows(g: Octree, pts: torch.Tensor, batch: torch.Tensor | None = None) -> torch.Tensor:
    rows = torch.empty(pts.shape[0], dtype=torch.int32, device=pts.device)
    _check(lib().oc_points_leaf_rows(_ptr(g.trees), _ptr(g.prefix), *g.dims(), _ptr(pts), _ptr(batch),
                                     pts.shape[0], _ptr(rows), _stream()), "oc_points_leaf_rows")
    return rows


def points_average(g: Octree, rows: torch.Tensor, feat: torch.Tensor) -> torch.Tensor:
    """[n_leaves, 1 + C]: occupancy flag and the mean point features per leaf."""
    c = feat.shape[1]
    out = torch.empty((g.n_leaves, c + 1), dtype=torch.float32, device=rows.device)
    ws = torch.empty(lib().oc_points_workspace(g.n_leaves, 1), dtype=torch.uint8, device=rows.device)
    _check(lib().oc_points_average(_ptr(rows), rows.shape[0], _ptr(feat), c, g.n_leaves, _ptr(out),
                                   _ptr(ws), ws.numel(), _stream()), "oc_points_average")
    return out


def points_vote(g: Octree, rows: torch.Tensor, labels: torch.Tensor, n_labels: int) -> torch.Tensor:
    """[n_leaves] majority label per leaf (-1 without points)."""
    out = torch.empty(g.n_leaves, dtype=torch.int32, device=rows.device)
    ws = torch.empty(lib().oc_points_workspace(g.n_leaves, n_labels), dtype=torch.uint8, device=rows.device)
    _check(lib().oc_points_vote(_ptr(rows), rows.shape[0], _ptr(labels), n_labels, g.n_leaves, _ptr(out),
                                _ptr(ws), ws.numel(), _stream()), "oc_points_vote")
    return out
