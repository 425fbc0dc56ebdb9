"""Python front-end of the CPU oracle for the grid-octree hot path.

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the benchmark's
CPU-baseline leg may import this module; the GPU library never does, and
this module imports nothing from the GPU library.  The arithmetic lives in
``octref.c`` (plain C, double precision, OpenMP over leaves); this file only
marshals numpy arrays.

Every function follows a passage of the OctNet paper (Riegler et al., CVPR
2017):

- ``data_idx_eq3`` / ``data_idx_bfs``: Eq. 3 and the breadth-first leaf order
  it counts (Sec. 3.1; supplement, "Data Index").
- ``build``: octree creation by splitting cells (Sec. 1, Sec. 3.1).
- ``oc2ten`` / ``ten2oc``: Eq. 4 and Eq. 5.
- ``conv3``: Eq. 8, i.e. ten2oc(avg) of the dense convolution of Eq. 7 applied
  to oc2ten of the input (the wrapper of Eq. 6).
- ``pool2_structure`` / ``pool2_max``: Eq. 10 (Sec. 3.2, "Pooling").
- ``unpool2_structure`` / ``unpool2``: Eq. 12 and the guided remark after it.
- ``conv3_bwd_data`` / ``conv3_bwd_weight`` / ``pool2_max_bwd`` /
  ``unpool2_bwd`` / ``relu_bwd``: the gradients of those maps (their
  adjoints: Eq. 8 is linear in the input and in the weights, Eq. 10 selects
  one input value per output value, Eq. 12 copies).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "octref.c")
_LIB = os.path.join(_HERE, "liboctref.so")

NBITS = 73
NNODES = 585


def build_library(force: bool = False) -> str:
    """Compile octref.c into liboctref.so with gcc (plain C, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build_library()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int, ctypes.c_long, ctypes.c_double
        sig = {
            "ocref_parent": (i32, [i32]),
            "ocref_child": (i32, [i32]),
            "ocref_bit": (i32, [P, i32]),
            "ocref_data_idx_eq3": (i64, [P, i32, i32, i32]),
            "ocref_data_idx_bfs": (i64, [P, i32, i32, i32, i32]),
            "ocref_tree_n_leaves": (i32, [P]),
            "ocref_tree_valid": (i32, [P]),
            "ocref_prefix": (None, [P, i64, P]),
            "ocref_leaf_info": (None, [P, i64, P, P]),
            "ocref_rowmap": (None, [P, P, i32, i32, i32, i32, P]),
            "ocref_build": (None, [P, i32, i32, i32, i32, i32, P]),
            "ocref_oc2ten": (None, [P, i64, P, i32, P]),
            "ocref_ten2oc": (None, [P, P, i32, i32, i32, i32, P, i32, i32, P]),
            "ocref_conv3": (None, [P, P, P, i32, i32, i32, i32, i32, P, i32, P, P, i32, i32, P, i64, P]),
            "ocref_dense_conv3": (None, [P, i32, i64, i64, i64, i32, P, i32, P]),
            "ocref_pool2_structure": (None, [P, i32, i32, i32, i32, P]),
            "ocref_pool2_max": (None, [P, P, i32, i32, i32, i32, P, i32, P, i64, P]),
            "ocref_unpool2_structure": (None, [P, i32, i32, i32, i32, P]),
            "ocref_unpool2": (None, [P, i32, i32, i32, P, i32, P, i64, P]),
            "ocref_relu": (None, [P, i64]),
            "ocref_conv3_bwd_data": (None, [P, P, i32, i32, i32, i32, P, i32, P, i32, i64, P]),
            "ocref_conv3_bwd_weight": (None, [P, P, i32, i32, i32, i32, P, i32, P, i32, i64, P, P]),
            "ocref_pool2_max_bwd": (None, [P, P, i32, i32, i32, i32, P, i32, P, i64, P, i64, P]),
            "ocref_unpool2_bwd": (None, [P, i32, i32, i32, i32, P, i64, P, i64, P]),
            "ocref_num_threads": (i32, []),
            "ocref_set_num_threads": (None, [i32]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return ctypes.c_void_p(a.ctypes.data)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ----------------------------------------------------------------------------
# Structure
# ----------------------------------------------------------------------------


@dataclass
class Grid:
    """A batch of N grids of gd x gh x gw shallow octrees.

    trees: uint32 [n_trees, 4] split bits (bit j in word j>>5, position j&31)
    prefix: int64 [n_trees + 1] leaves of all earlier trees
    """

    n: int
    gd: int
    gh: int
    gw: int
    trees: np.ndarray
    prefix: np.ndarray

    @property
    def n_trees(self) -> int:
        return self.n * self.gd * self.gh * self.gw

    @property
    def n_leaves(self) -> int:
        return int(self.prefix[-1])

    @property
    def dense_shape(self):
        return (self.n, 8 * self.gd, 8 * self.gh, 8 * self.gw)


def parent(i: int) -> int:
    """Eq. 1."""
    return lib().ocref_parent(int(i))


def child(i: int) -> int:
    """Eq. 2."""
    return lib().ocref_child(int(i))


def bit(tree_words, i: int) -> int:
    t = _c(tree_words, np.uint32)
    return lib().ocref_bit(_p(t), int(i))


def data_idx_eq3(bits01, b: int, i: int) -> int:
    """Eq. 3 for branching factor b (8: octree; 4: the supplement's quadtree)."""
    a = _c(bits01, np.uint8)
    return lib().ocref_data_idx_eq3(_p(a), len(a), int(b), int(i))


def data_idx_bfs(bits01, b: int, maxdepth: int, i: int) -> int:
    """Rank of leaf i in breadth-first order, by enumeration (-1: not a leaf)."""
    a = _c(bits01, np.uint8)
    return lib().ocref_data_idx_bfs(_p(a), len(a), int(b), int(maxdepth), int(i))


def tree_n_leaves(tree_words) -> int:
    t = _c(tree_words, np.uint32)
    return lib().ocref_tree_n_leaves(_p(t))


def tree_valid(tree_words) -> bool:
    t = _c(tree_words, np.uint32)
    return bool(lib().ocref_tree_valid(_p(t)))


def words_to_bits(tree_words) -> np.ndarray:
    """uint32[4] -> uint8[73] (bit j of the split string)."""
    w = _c(tree_words, np.uint32)
    return np.array([(int(w[j >> 5]) >> (j & 31)) & 1 for j in range(NBITS)], dtype=np.uint8)


def bits_to_words(bits01) -> np.ndarray:
    w = np.zeros(4, dtype=np.uint32)
    for j, b in enumerate(bits01):
        if b:
            w[j >> 5] |= np.uint32(1 << (j & 31))
    return w


def prefix_of(trees: np.ndarray) -> np.ndarray:
    trees = _c(trees, np.uint32).reshape(-1, 4)
    out = np.zeros(trees.shape[0] + 1, dtype=np.int64)
    lib().ocref_prefix(_p(trees), trees.shape[0], _p(out))
    return out


def build(occ: np.ndarray, rule: str = "mixed") -> Grid:
    """Split every node whose occupancy is mixed (rule 'mixed') or non-empty
    (rule 'any'); occ is uint8 [N, 8gd, 8gh, 8gw]."""
    occ = _c(occ, np.uint8)
    n, D, H, W = occ.shape
    assert D % 8 == 0 and H % 8 == 0 and W % 8 == 0
    gd, gh, gw = D // 8, H // 8, W // 8
    trees = np.zeros((n * gd * gh * gw, 4), dtype=np.uint32)
    lib().ocref_build(_p(occ), n, gd, gh, gw, 0 if rule == "mixed" else 1, _p(trees))
    return Grid(n, gd, gh, gw, trees, prefix_of(trees))


def make_grid(trees: np.ndarray, n: int, gd: int, gh: int, gw: int) -> Grid:
    trees = _c(trees, np.uint32).reshape(-1, 4)
    assert trees.shape[0] == n * gd * gh * gw
    return Grid(n, gd, gh, gw, trees, prefix_of(trees))


def leaf_info(g: Grid) -> np.ndarray:
    """uint64 [n_leaves]: tree << 10 | bit index of every leaf, in row order."""
    out = np.zeros(g.n_leaves, dtype=np.uint64)
    lib().ocref_leaf_info(_p(g.trees), g.n_trees, _p(g.prefix), _p(out))
    return out


def rowmap(g: Grid) -> np.ndarray:
    """int64 [N, 8gd, 8gh, 8gw]: row of the leaf containing each voxel."""
    out = np.zeros(g.dense_shape, dtype=np.int64)
    lib().ocref_rowmap(_p(g.trees), _p(g.prefix), g.n, g.gd, g.gh, g.gw, _p(out))
    return out


def rowmap_sample(g: Grid, s: int) -> np.ndarray:
    """rowmap of sample s alone (rows stay global)."""
    per = g.gd * g.gh * g.gw
    sub = Grid(1, g.gd, g.gh, g.gw, g.trees[s * per:(s + 1) * per], g.prefix[s * per:(s + 1) * per + 1])
    out = np.zeros((1,) + g.dense_shape[1:], dtype=np.int64)
    lib().ocref_rowmap(_p(sub.trees), _p(np.ascontiguousarray(sub.prefix)), 1, g.gd, g.gh, g.gw, _p(out))
    return out[0]


# ----------------------------------------------------------------------------
# Features
# ----------------------------------------------------------------------------


def oc2ten(g: Grid, data: np.ndarray, rm: np.ndarray | None = None) -> np.ndarray:
    """Eq. 4: dense NDHWC tensor (float64)."""
    data = _c(data, np.float64)
    c = data.shape[1]
    rm = rowmap(g) if rm is None else _c(rm, np.int64)
    out = np.zeros(g.dense_shape + (c,), dtype=np.float64)
    lib().ocref_oc2ten(_p(rm), rm.size, _p(data), c, _p(out))
    return out


def ten2oc(g: Grid, dense: np.ndarray, pool: str = "avg") -> np.ndarray:
    """Eq. 5: leaf features [n_leaves, C] (float64); pool 'avg' or 'max'."""
    dense = _c(dense, np.float64)
    assert dense.shape[:4] == g.dense_shape
    c = dense.shape[4]
    out = np.zeros((g.n_leaves, c), dtype=np.float64)
    lib().ocref_ten2oc(_p(g.trees), _p(g.prefix), g.n, g.gd, g.gh, g.gw, _p(dense), c,
                       0 if pool == "avg" else 1, _p(out))
    return out


def conv3(g: Grid, data: np.ndarray, w: np.ndarray, bias=None, relu: bool = False,
          rows=None, info=None, rm=None, rm_sample: int = -1) -> np.ndarray:
    """Eq. 8: grid-octree 3x3x3 convolution with average pooling, evaluated
    leaf by leaf as ten2oc(conv_dense(oc2ten(O))) restricted to each leaf's
    cell.  w is [Cout, Cin, 3, 3, 3] in Eq. 7's orientation.  ``rows`` selects
    a subset of leaves (default: all); the result is [len(rows), Cout].
    ``rm`` is rowmap(g) (all samples), or rowmap_sample(g, rm_sample)."""
    data = _c(data, np.float64)
    w = _c(w, np.float64)
    cout, cin = w.shape[0], w.shape[1]
    assert data.shape[1] == cin and w.shape[2:] == (3, 3, 3)
    b = None if bias is None else _c(bias, np.float64)
    info = leaf_info(g) if info is None else _c(info, np.uint64)
    if rows is None:
        rows = np.arange(g.n_leaves, dtype=np.int64)
    rows = _c(rows, np.int64)
    out = np.zeros((rows.size, cout), dtype=np.float64)
    if rows.size == 0:
        return out
    if rm is None:
        rm = rowmap(g) if rm_sample < 0 else rowmap_sample(g, rm_sample)
    rm = _c(rm, np.int64)
    assert rm.shape == (g.dense_shape if rm_sample < 0 else g.dense_shape[1:])
    lib().ocref_conv3(_p(g.trees), _p(info), _p(rm), int(rm_sample), g.n, g.gd, g.gh, g.gw,
                      _p(data), cin, _p(w), _p(b) if b is not None else None, cout,
                      int(bool(relu)), _p(rows), rows.size, _p(out))
    return out


def conv3_sampled(g: Grid, data: np.ndarray, w: np.ndarray, bias, relu: bool, rows,
                  info=None) -> np.ndarray:
    """conv3 on a subset of rows, building the rowmap one sample at a time so
    that large batches never hold every sample's dense map at once."""
    info = leaf_info(g) if info is None else info
    rows = np.asarray(rows, dtype=np.int64)
    per = g.gd * g.gh * g.gw
    samples = (info[rows] >> np.uint64(10)).astype(np.int64) // per
    out = np.zeros((rows.size, w.shape[0]), dtype=np.float64)
    for s in np.unique(samples):
        sel = np.nonzero(samples == s)[0]
        out[sel] = conv3(g, data, w, bias, relu, rows=rows[sel], info=info,
                         rm=rowmap_sample(g, int(s)), rm_sample=int(s))
    return out


def dense_conv3(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Eq. 7 over a whole NDHWC tensor with zero padding 1 (float64)."""
    x = _c(x, np.float64)
    w = _c(w, np.float64)
    n, D, H, W, cin = x.shape
    cout = w.shape[0]
    y = np.zeros((n, D, H, W, cout), dtype=np.float64)
    lib().ocref_dense_conv3(_p(x), n, D, H, W, cin, _p(w), cout, _p(y))
    return y


def conv3_wrapped(g: Grid, data: np.ndarray, w: np.ndarray, bias=None, relu=False) -> np.ndarray:
    """Eq. 6 literally: ten2oc_avg(dense_conv3(oc2ten(O))) + bias (tiny grids)."""
    y = ten2oc(g, dense_conv3(oc2ten(g, data), w), "avg")
    if bias is not None:
        y = y + np.asarray(bias, dtype=np.float64)[None, :]
    if relu:
        y = np.maximum(y, 0.0)
    return y


# ----------------------------------------------------------------------------
# Pool / unpool
# ----------------------------------------------------------------------------


def pool2_structure(g: Grid) -> Grid:
    assert g.gd % 2 == 0 and g.gh % 2 == 0 and g.gw % 2 == 0
    out = np.zeros((g.n * (g.gd // 2) * (g.gh // 2) * (g.gw // 2), 4), dtype=np.uint32)
    lib().ocref_pool2_structure(_p(g.trees), g.n, g.gd, g.gh, g.gw, _p(out))
    return make_grid(out, g.n, g.gd // 2, g.gh // 2, g.gw // 2)


def pool2_max(g: Grid, data: np.ndarray, out_g: Grid | None = None, rows=None) -> tuple[Grid, np.ndarray]:
    """Eq. 10: returns (output structure, output data); ``rows`` restricts the
    data to a subset of output rows."""
    data = _c(data, np.float64)
    c = data.shape[1]
    out_g = pool2_structure(g) if out_g is None else out_g
    info_in = leaf_info(g)
    info_out = leaf_info(out_g)
    if rows is not None:
        info_out = _c(info_out[np.asarray(rows, dtype=np.int64)], np.uint64)
    rm = rowmap(g)
    out = np.zeros((info_out.size, c), dtype=np.float64)
    lib().ocref_pool2_max(_p(info_in), _p(rm), g.n, g.gd, g.gh, g.gw, _p(data), c,
                          _p(info_out), info_out.size, _p(out))
    return out_g, out


def unpool2_structure(g: Grid) -> Grid:
    out = np.zeros((g.n * 8 * g.gd * g.gh * g.gw, 4), dtype=np.uint32)
    lib().ocref_unpool2_structure(_p(g.trees), g.n, g.gd, g.gh, g.gw, _p(out))
    return make_grid(out, g.n, 2 * g.gd, 2 * g.gh, 2 * g.gw)


def unpool2(g: Grid, data: np.ndarray, guide: Grid | None = None, rows=None) -> tuple[Grid, np.ndarray]:
    """Eq. 12 (guide None) or the guided variant: returns (structure, data);
    ``rows`` restricts the data to a subset of output rows."""
    data = _c(data, np.float64)
    c = data.shape[1]
    if guide is None:
        out_g = unpool2_structure(g)
    else:
        assert (guide.n, guide.gd, guide.gh, guide.gw) == (g.n, 2 * g.gd, 2 * g.gh, 2 * g.gw)
        out_g = guide
    info_out = leaf_info(out_g)
    if rows is not None:
        info_out = _c(info_out[np.asarray(rows, dtype=np.int64)], np.uint64)
    rm = rowmap(g)
    out = np.zeros((info_out.size, c), dtype=np.float64)
    lib().ocref_unpool2(_p(rm), g.gd, g.gh, g.gw, _p(data), c, _p(info_out), info_out.size, _p(out))
    return out_g, out


def relu(x: np.ndarray) -> np.ndarray:
    y = np.array(x, dtype=np.float64, copy=True, order="C")
    lib().ocref_relu(_p(y), y.size)
    return y


def num_threads() -> int:
    return lib().ocref_num_threads()


def set_num_threads(n: int) -> None:
    lib().ocref_set_num_threads(int(n))


# ----------------------------------------------------------------------------
# Gradients
# ----------------------------------------------------------------------------


def conv3_bwd_data(g: Grid, dy: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Input gradient of Eq. 8 (bias and ReLU excluded): [n_leaves, Cin]."""
    dy = _c(dy, np.float64)
    w = _c(w, np.float64)
    cout, cin = w.shape[0], w.shape[1]
    assert dy.shape == (g.n_leaves, cout)
    info, rm = leaf_info(g), rowmap(g)
    dx = np.zeros((g.n_leaves, cin), dtype=np.float64)
    lib().ocref_conv3_bwd_data(_p(info), _p(rm), g.n, g.gd, g.gh, g.gw, _p(dy), cout, _p(w),
                               cin, g.n_leaves, _p(dx))
    return dx


def conv3_bwd_weight(g: Grid, x: np.ndarray, dy: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Weight and bias gradients of Eq. 8: ([Cout, Cin, 3, 3, 3], [Cout])."""
    x = _c(x, np.float64)
    dy = _c(dy, np.float64)
    cin, cout = x.shape[1], dy.shape[1]
    assert x.shape[0] == g.n_leaves and dy.shape[0] == g.n_leaves
    info, rm = leaf_info(g), rowmap(g)
    dw = np.zeros((cout, cin, 3, 3, 3), dtype=np.float64)
    db = np.zeros(cout, dtype=np.float64)
    lib().ocref_conv3_bwd_weight(_p(info), _p(rm), g.n, g.gd, g.gh, g.gw, _p(x), cin, _p(dy),
                                 cout, g.n_leaves, _p(dw), _p(db))
    return dw, db


def pool2_max_bwd(g: Grid, x: np.ndarray, dy: np.ndarray, out_g: Grid | None = None) -> np.ndarray:
    """Gradient of Eq. 10 with respect to the input leaves: [n_leaves(g), C]."""
    x = _c(x, np.float64)
    dy = _c(dy, np.float64)
    c = x.shape[1]
    out_g = pool2_structure(g) if out_g is None else out_g
    info_in, info_out, rm = leaf_info(g), leaf_info(out_g), rowmap(g)
    assert dy.shape == (out_g.n_leaves, c)
    dx = np.zeros((g.n_leaves, c), dtype=np.float64)
    lib().ocref_pool2_max_bwd(_p(info_in), _p(rm), g.n, g.gd, g.gh, g.gw, _p(x), c, _p(info_out),
                              info_out.size, _p(dy), g.n_leaves, _p(dx))
    return dx


def unpool2_bwd(g: Grid, dy: np.ndarray, out_g: Grid) -> np.ndarray:
    """Gradient of Eq. 12 (plain or guided; out_g is the output structure)
    with respect to the input leaves: [n_leaves(g), C]."""
    dy = _c(dy, np.float64)
    c = dy.shape[1]
    info_out, rm = leaf_info(out_g), rowmap(g)
    assert dy.shape[0] == out_g.n_leaves
    dx = np.zeros((g.n_leaves, c), dtype=np.float64)
    lib().ocref_unpool2_bwd(_p(rm), g.gd, g.gh, g.gw, c, _p(info_out), info_out.size, _p(dy),
                            g.n_leaves, _p(dx))
    return dx


def concat(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Skip connection of the segmentation network (architecture table):
    the channels of a followed by those of b, row by row (one structure)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape[0] == b.shape[0]
    return np.concatenate([a, b], axis=1)


def concat_bwd(d: np.ndarray, ca: int) -> tuple[np.ndarray, np.ndarray]:
    """Gradient of concat: the first ca channels of d, and the rest."""
    d = np.asarray(d, dtype=np.float64)
    return d[:, :ca].copy(), d[:, ca:].copy()


def points_voxelize(pts: np.ndarray, batch, n: int, gd: int, gh: int, gw: int) -> np.ndarray:
    """Sec. 5: a point cloud mapped into the voxel grid; a point lies in voxel
    floor(coordinate); points outside the grid (or the batch) are dropped."""
    pts = np.asarray(pts, dtype=np.float32)
    b = np.zeros(len(pts), np.int64) if batch is None else np.asarray(batch, np.int64)
    D, H, W = 8 * gd, 8 * gh, 8 * gw
    occ = np.zeros((n, D, H, W), dtype=np.uint8)
    ok = point_inside(pts, b, n, D, H, W)
    v = np.floor(pts[ok]).astype(np.int64)
    occ[b[ok], v[:, 0], v[:, 1], v[:, 2]] = 1
    return occ


def point_inside(pts, b, n, D, H, W):
    lim = np.array([D, H, W], dtype=np.float32)
    return np.all(pts >= 0, axis=1) & np.all(pts < lim, axis=1) & (b >= 0) & (b < n)


def points_leaf_rows(g: Grid, pts: np.ndarray, batch) -> np.ndarray:
    """The row of the leaf whose cell holds each point (-1 if dropped), read
    from the dense row map of the structure."""
    pts = np.asarray(pts, dtype=np.float32)
    b = np.zeros(len(pts), np.int64) if batch is None else np.asarray(batch, np.int64)
    ok = point_inside(pts, b, g.n, 8 * g.gd, 8 * g.gh, 8 * g.gw)
    rows = np.full(len(pts), -1, dtype=np.int64)
    v = np.floor(pts[ok]).astype(np.int64)
    rm = rowmap(g)
    rows[ok] = rm[b[ok], v[:, 0], v[:, 1], v[:, 2]]
    return rows


def points_average(n_leaves: int, rows: np.ndarray, feat: np.ndarray) -> np.ndarray:
    """Sec. 5: a leaf holding points takes the mean of their features; channel
    0 is the binary occupancy (1 where a point fell in the leaf)."""
    rows = np.asarray(rows, np.int64)
    feat = np.asarray(feat, np.float64)
    c = feat.shape[1]
    out = np.zeros((n_leaves, c + 1), dtype=np.float64)
    cnt = np.zeros(n_leaves, dtype=np.int64)
    ok = rows >= 0
    np.add.at(out[:, 1:], rows[ok], feat[ok])
    np.add.at(cnt, rows[ok], 1)
    has = cnt > 0
    out[has, 1:] /= cnt[has, None]
    out[has, 0] = 1.0
    return out


def points_vote(n_leaves: int, rows: np.ndarray, labels: np.ndarray, n_labels: int) -> np.ndarray:
    """Sec. 5: the majority label of a leaf's points (the smallest of tied
    labels; -1 without labelled points)."""
    rows = np.asarray(rows, np.int64)
    labels = np.asarray(labels, np.int64)
    hist = np.zeros((n_leaves, n_labels), dtype=np.int64)
    ok = (rows >= 0) & (labels >= 0) & (labels < n_labels)
    np.add.at(hist, (rows[ok], labels[ok]), 1)
    out = np.where(hist.max(axis=1) > 0, hist.argmax(axis=1), -1)
    return out.astype(np.int64)


def relu_bwd(y: np.ndarray, dy: np.ndarray) -> np.ndarray:
    """Gradient of max(0, .) given its output y: dy where y > 0, else 0."""
    y = np.asarray(y, dtype=np.float64)
    return np.where(y > 0.0, np.asarray(dy, dtype=np.float64), 0.0)
