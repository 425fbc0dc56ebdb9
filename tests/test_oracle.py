"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: values the
paper prints, closed forms, invariants, brute force on tiny inputs, and
textbook library routines (torch CPU conv3d / max_pool3d) that the oracle
does not call.
"""
import os

import numpy as np
import pytest
import torch

import octref as O
from paper_1611_05009_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, v = [x.strip() for x in line.split("=", 1)]
            vals[k] = v
    return vals


def _bits_from_string(s):
    return np.array([int(c) for c in s.replace(" ", "")], dtype=np.uint8)


# ----------------------------------------------------------------------------
# Bit strings and the data index (Sec. 3.1, Eq. 1-3, supplement "Data Index")
# ----------------------------------------------------------------------------


def test_parent_child_closed_forms_exhaustive():
    # Every node i >= 1 lies among the 8 children of its parent (Eq. 1, 2).
    for i in range(1, 585):
        p = O.parent(i)
        assert O.child(p) <= i < O.child(p) + 8
    # Children of every internal node map back to it.
    for i in range(0, 73):
        for k in range(8):
            assert O.parent(O.child(i) + k) == i
    # Depth boundaries: nodes 1..8 are depth 1, 9..72 depth 2, 73..584 depth 3.
    assert O.child(0) == 1 and O.child(8) + 7 == 72 and O.child(72) + 7 == 584


def test_quadtree_worked_example():
    g = _read_golden("quadtree_data_idx.txt")
    bits = _bits_from_string(g["bits"])
    b, i = int(g["branching"]), int(g["i"])
    assert len(bits) == 21
    pa = (i - 1) // b
    assert pa == int(g["parent"])
    assert b * int(bits[:pa].sum()) + 1 == int(g["nodes_above"])
    assert int(bits[:i].sum()) == int(g["split_before"])
    assert (i - 1) % b == int(g["offset"])
    assert O.data_idx_eq3(bits, b, i) == int(g["data_idx"])
    assert O.data_idx_bfs(bits, b, int(g["max_depth"]), i) == int(g["data_idx"])


def test_quadtree_eq3_matches_bfs_for_every_leaf():
    g = _read_golden("quadtree_data_idx.txt")
    bits = _bits_from_string(g["bits"])
    leaves = [i for i in range(85) if O.data_idx_bfs(bits, 4, 3, i) >= 0]
    assert len(leaves) == 1 + 3 * int(bits.sum())
    for i in leaves:
        assert O.data_idx_eq3(bits, 4, i) == O.data_idx_bfs(bits, 4, 3, i)
    assert sorted(O.data_idx_bfs(bits, 4, 3, i) for i in leaves) == list(range(len(leaves)))


def test_fig3_octree_string():
    g = _read_golden("fig3_octree_bits.txt")
    bits = np.zeros(73, dtype=np.uint8)
    s = _bits_from_string(g["bits"])
    bits[: len(s)] = s
    assert sorted(np.nonzero(bits)[0].tolist()) == [int(x) for x in g["split_bits"].split()]
    words = O.bits_to_words(bits)
    assert O.tree_valid(words)
    assert O.tree_n_leaves(words) == int(g["n_leaves"])
    leaves = [i for i in range(585) if O.data_idx_bfs(bits, 8, 3, i) >= 0]
    assert len(leaves) == int(g["n_leaves"])
    for i in leaves:
        assert O.data_idx_eq3(bits, 8, i) == O.data_idx_bfs(bits, 8, 3, i)


def _random_tree(rng, p1=0.5, p2=0.4):
    bits = np.zeros(73, dtype=np.uint8)
    if rng.random() < 0.9:
        bits[0] = 1
        for o in range(8):
            if rng.random() < p1:
                bits[1 + o] = 1
                for q in range(8):
                    bits[9 + 8 * o + q] = rng.random() < p2
    return bits


def test_eq3_equals_bfs_rank_on_random_trees():
    rng = np.random.default_rng(5)
    for _ in range(150):
        bits = _random_tree(rng)
        words = O.bits_to_words(bits)
        assert O.tree_valid(words)
        n = O.tree_n_leaves(words)
        assert n == 1 + 7 * int(bits.sum()) and n <= 512
        ranks = []
        for i in range(585):
            r = O.data_idx_bfs(bits, 8, 3, i)
            if r >= 0:
                assert O.data_idx_eq3(bits, 8, i) == r
                ranks.append(r)
        assert sorted(ranks) == list(range(n))


def test_tree_valid_rejects_orphan_bits():
    bits = np.zeros(73, dtype=np.uint8)
    bits[9] = 1  # child of node 1, which is not split
    assert not O.tree_valid(O.bits_to_words(bits))
    w = np.zeros(4, dtype=np.uint32)
    w[2] = 1 << 9  # bit 73 is beyond the string
    assert not O.tree_valid(w)


# ----------------------------------------------------------------------------
# Build (octree creation by splitting), oc2ten, ten2oc
# ----------------------------------------------------------------------------


def _node_regions():
    """(bit index, depth, origin, size) of all 73 internal nodes, by brute
    force over the octant paths."""
    out = []
    for i in range(73):
        path, j = [], i
        while j > 0:
            path.append((j - 1) % 8)
            j = (j - 1) // 8
        s, o = 8, [0, 0, 0]
        for oc in reversed(path):
            s //= 2
            o = [o[0] + ((oc >> 2) & 1) * s, o[1] + ((oc >> 1) & 1) * s, o[2] + (oc & 1) * s]
        out.append((i, len(path), o, s))
    return out


@pytest.mark.parametrize("rule", ["mixed", "any"])
def test_build_split_rule_brute_force(rule):
    rng = np.random.default_rng(11)
    occ = synth.random_occupancy(rng, 2, 2, 3, 2)
    g = O.build(occ, rule)
    regions = _node_regions()
    for t in range(g.n_trees):
        s_, rem = divmod(t, g.gd * g.gh * g.gw)
        td, rem = divmod(rem, g.gh * g.gw)
        th, tw = divmod(rem, g.gw)
        cube = occ[s_, 8 * td:8 * td + 8, 8 * th:8 * th + 8, 8 * tw:8 * tw + 8]
        bits = O.words_to_bits(g.trees[t])
        assert O.tree_valid(g.trees[t])
        for i, dep, o, s in regions:
            exists = i == 0 or bits[(i - 1) // 8]
            reg = cube[o[0]:o[0] + s, o[1]:o[1] + s, o[2]:o[2] + s]
            want = (reg.any() and not reg.all()) if rule == "mixed" else reg.any()
            assert bits[i] == (bool(exists) and bool(want)), (t, i)


def test_build_is_lossless_and_leaves_homogeneous():
    rng = np.random.default_rng(3)
    occ = synth.random_occupancy(rng, 2, 3, 2, 2)
    g = O.build(occ)
    occ_leaf = O.ten2oc(g, occ[..., None].astype(np.float64), "avg")
    # every leaf is homogeneous: the average is exactly 0 or 1
    assert np.all((occ_leaf == 0.0) | (occ_leaf == 1.0))
    assert np.array_equal(O.oc2ten(g, occ_leaf)[..., 0], occ.astype(np.float64))
    assert g.n_leaves == sum(1 + 7 * int(O.words_to_bits(t).sum()) for t in g.trees)


def test_oc2ten_ten2oc_round_trip_and_max():
    rng = np.random.default_rng(4)
    g = O.build(synth.random_occupancy(rng, 1, 2, 2, 2))
    data = rng.standard_normal((g.n_leaves, 3))
    dense = O.oc2ten(g, data)
    # averaging s^3 equal copies rounds only in the last bits of a double
    np.testing.assert_allclose(O.ten2oc(g, dense, "avg"), data, rtol=1e-14, atol=0)
    assert np.array_equal(O.ten2oc(g, dense, "max"), data)
    # ten2oc of an arbitrary tensor: brute force per leaf
    x = rng.standard_normal(g.dense_shape + (2,))
    info = O.leaf_info(g)
    avg, mx = O.ten2oc(g, x, "avg"), O.ten2oc(g, x, "max")
    regions = {i: (o, s) for i, _, o, s in _node_regions()}
    for r in rng.choice(g.n_leaves, size=50, replace=False):
        t, bit = int(info[r]) >> 10, int(info[r]) & 1023
        td, rem = divmod(t, g.gh * g.gw)
        th, tw = divmod(rem, g.gw)
        if bit >= 73:
            p = (bit - 1) // 8
            (o, s) = regions[p]
            oc = (bit - 1) % 8
            o = [o[0] + ((oc >> 2) & 1), o[1] + ((oc >> 1) & 1), o[2] + (oc & 1)]
            s = 1
        else:
            o, s = regions[bit]
        cell = x[0, 8 * td + o[0]:8 * td + o[0] + s, 8 * th + o[1]:8 * th + o[1] + s,
                 8 * tw + o[2]:8 * tw + o[2] + s]
        np.testing.assert_allclose(avg[r], cell.reshape(-1, 2).mean(0), rtol=1e-12, atol=1e-12)
        np.testing.assert_array_equal(mx[r], cell.reshape(-1, 2).max(0))


def test_leaf_info_rows_are_concatenated_in_tree_order():
    rng = np.random.default_rng(9)
    g = O.build(synth.random_occupancy(rng, 2, 2, 2, 1))
    info = O.leaf_info(g)
    trees = (info >> np.uint64(10)).astype(np.int64)
    assert np.all(np.diff(trees) >= 0)
    for t in range(g.n_trees):
        rows = np.nonzero(trees == t)[0]
        assert rows[0] == g.prefix[t] and rows.size == g.prefix[t + 1] - g.prefix[t]
        bits = O.words_to_bits(g.trees[t])
        for k, r in enumerate(rows):
            assert O.data_idx_eq3(bits, 8, int(info[r]) & 1023) == k


# ----------------------------------------------------------------------------
# Convolution (Eq. 7, Eq. 8)
# ----------------------------------------------------------------------------


def _torch_conv_dense(x_ndhwc, w):
    """Eq. 7 by a textbook routine: torch's conv3d is a cross-correlation, so
    Eq. 7's true convolution uses the kernel flipped along all three axes."""
    x = torch.from_numpy(np.ascontiguousarray(x_ndhwc)).permute(0, 4, 1, 2, 3)
    wt = torch.from_numpy(np.ascontiguousarray(w)).flip(2, 3, 4)
    y = torch.nn.functional.conv3d(x, wt, padding=1)
    return y.permute(0, 2, 3, 4, 1).contiguous().numpy()


@pytest.mark.parametrize("seed,cin,cout", [(0, 1, 2), (1, 3, 4), (2, 5, 3)])
def test_conv_matches_textbook_conv3d_wrapped(seed, cin, cout):
    rng = np.random.default_rng(100 + seed)
    g = O.build(synth.random_occupancy(rng, 2, 2, 2, 3))
    data = rng.standard_normal((g.n_leaves, cin))
    w = rng.standard_normal((cout, cin, 3, 3, 3))
    b = rng.standard_normal(cout)
    want = O.ten2oc(g, _torch_conv_dense(O.oc2ten(g, data), w), "avg") + b
    got = O.conv3(g, data, w, b)
    np.testing.assert_allclose(got, want, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(O.conv3_wrapped(g, data, w, b), want, rtol=1e-11, atol=1e-11)
    # ReLU variant and the per-sample evaluation agree too
    rows = rng.choice(g.n_leaves, size=40, replace=False)
    np.testing.assert_allclose(O.conv3_sampled(g, data, w, b, True, rows),
                               np.maximum(want[rows], 0), rtol=1e-11, atol=1e-11)


def test_conv_kernel_orientation_is_eq7():
    # Fully split tree (every leaf one voxel), input 1 at voxel (4,4,4) only,
    # delta kernel at tap (l,m,n) = (0,1,1): Eq. 7 gives T[i,j,k] = x[i+1,j,k],
    # so the response appears one voxel *below* the input along d.
    g = O.build(np.ones((1, 8, 8, 8), dtype=np.uint8), "any")
    x = np.zeros((1, 8, 8, 8, 1))
    x[0, 4, 4, 4, 0] = 1.0
    data = O.ten2oc(g, x, "avg")
    w = np.zeros((1, 1, 3, 3, 3))
    w[0, 0, 0, 1, 1] = 1.0
    y = O.oc2ten(g, O.conv3(g, data, w))[0, ..., 0]
    assert y[3, 4, 4] == 1.0 and y.sum() == 1.0


def test_conv_fully_split_equals_dense():
    rng = np.random.default_rng(7)
    occ = np.ones((1, 16, 8, 8), dtype=np.uint8)
    g = O.build(occ, "any")  # every node split: all leaves are single voxels
    assert g.n_leaves == 16 * 8 * 8
    data = rng.standard_normal((g.n_leaves, 2))
    w = rng.standard_normal((3, 2, 3, 3, 3))
    dense_in = O.oc2ten(g, data)
    want = _torch_conv_dense(dense_in, w)
    got = O.oc2ten(g, O.conv3(g, data, w))
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_conv_single_cell_closed_form():
    # One unsplit tree, x = 1, all-ones kernel, zero padding: each axis sums
    # 6*3 + 2*2 = 22 over the 8 voxels, so the cell average is 22^3 / 512.
    g = O.build(np.zeros((1, 8, 8, 8), dtype=np.uint8))
    assert g.n_leaves == 1
    y = O.conv3(g, np.ones((1, 1)), np.ones((1, 1, 3, 3, 3)))
    assert y[0, 0] == 22.0 ** 3 / 512.0 == 20.796875


def test_conv_delta_kernel_is_identity():
    rng = np.random.default_rng(8)
    g = O.build(synth.random_occupancy(rng, 1, 2, 2, 2))
    data = rng.standard_normal((g.n_leaves, 3))
    w = np.zeros((3, 3, 3, 3, 3))
    for c in range(3):
        w[c, c, 1, 1, 1] = 1.0
    np.testing.assert_allclose(O.conv3(g, data, w), data, rtol=1e-14, atol=1e-15)


def test_conv_linearity():
    rng = np.random.default_rng(12)
    g = O.build(synth.random_occupancy(rng, 1, 2, 2, 2))
    x1, x2 = rng.standard_normal((2, g.n_leaves, 2))
    w1, w2 = rng.standard_normal((2, 3, 2, 3, 3, 3))
    np.testing.assert_allclose(O.conv3(g, 2 * x1 - x2, w1),
                               2 * O.conv3(g, x1, w1) - O.conv3(g, x2, w1), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(O.conv3(g, x1, w1 + 3 * w2),
                               O.conv3(g, x1, w1) + 3 * O.conv3(g, x1, w2), rtol=1e-10, atol=1e-10)


def test_conv_is_a_sum_over_input_channel_blocks():
    """Eq. 7 sums over input channels: the convolution of all channels is
    the sum of the convolutions of channel blocks with the matching weight
    columns, and output channels are independent (the identity the wide
    layers' channel blocks rest on)."""
    rng = np.random.default_rng(14)
    g = O.build(synth.random_occupancy(rng, 1, 2, 2, 2))
    cin, cout = 6, 4
    x = rng.standard_normal((g.n_leaves, cin))
    w = rng.standard_normal((cout, cin, 3, 3, 3))
    full = O.conv3(g, x, w)
    parts = sum(O.conv3(g, x[:, j:j + 2], w[:, j:j + 2]) for j in range(0, cin, 2))
    np.testing.assert_allclose(parts, full, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(O.conv3(g, x, w[1:3]), full[:, 1:3], rtol=1e-12, atol=1e-12)


def test_conv_axis_permutation_equivariance():
    rng = np.random.default_rng(13)
    occ = synth.random_occupancy(rng, 1, 1, 2, 3)
    g = O.build(occ)
    x = rng.standard_normal(g.dense_shape + (2,))
    data = O.ten2oc(g, x, "avg")
    w = rng.standard_normal((2, 2, 3, 3, 3))
    y = O.oc2ten(g, O.conv3(g, data, w))
    perm = (2, 0, 1)  # new axes (d,h,w) = old (w,d,h)
    occ_p = np.ascontiguousarray(occ.transpose((0,) + tuple(p + 1 for p in perm)))
    gp = O.build(occ_p)
    xp = O.oc2ten(g, data).transpose((0,) + tuple(p + 1 for p in perm) + (4,))
    dp = O.ten2oc(gp, xp, "avg")
    wp = np.ascontiguousarray(w.transpose((0, 1) + tuple(p + 2 for p in perm)))
    yp = O.oc2ten(gp, O.conv3(gp, dp, wp))
    np.testing.assert_allclose(yp, y.transpose((0,) + tuple(p + 1 for p in perm) + (4,)),
                               rtol=1e-11, atol=1e-11)


def test_conv_tree_translation_equivariance():
    # An object in tree (1,1,1) of a 4^3-tree grid, moved by whole trees to
    # (2,1,2): the response around it moves with it (its 26 neighbour trees
    # are empty in both grids).
    rng = np.random.default_rng(14)
    occ = np.zeros((1, 32, 32, 32), dtype=np.uint8)
    occ[0, 8:16, 8:16, 8:16] = synth.random_occupancy(rng, 1, 1, 1, 1, density=0.2)[0]
    shifted = np.zeros_like(occ)
    shifted[0, 16:24, 8:16, 16:24] = occ[0, 8:16, 8:16, 8:16]
    g, gs = O.build(occ), O.build(shifted)
    x = rng.standard_normal(g.dense_shape + (1,)) * (occ[..., None] > 0)
    xs = np.zeros_like(x)
    xs[0, 16:24, 8:16, 16:24] = x[0, 8:16, 8:16, 8:16]
    w = rng.standard_normal((2, 1, 3, 3, 3))
    y = O.oc2ten(g, O.conv3(g, O.ten2oc(g, x), w))
    ys = O.oc2ten(gs, O.conv3(gs, O.ten2oc(gs, xs), w))
    np.testing.assert_allclose(ys[:, 8:32, 0:24, 8:32], y[:, 0:24, 0:24, 0:24], rtol=1e-11, atol=1e-11)


# ----------------------------------------------------------------------------
# Pooling (Eq. 9, Eq. 10) and unpooling (Eq. 11, Eq. 12, guided remark)
# ----------------------------------------------------------------------------


def _leaf_cells(g):
    """Set of (sample, global origin, size) of every leaf, by brute force."""
    regions = {i: (o, s) for i, _, o, s in _node_regions()}
    cells = set()
    for r, v in enumerate(O.leaf_info(g)):
        t, bit = int(v) >> 10, int(v) & 1023
        smp, rem = divmod(t, g.gd * g.gh * g.gw)
        td, rem = divmod(rem, g.gh * g.gw)
        th, tw = divmod(rem, g.gw)
        if bit >= 73:
            o, _ = regions[(bit - 1) // 8]
            oc = (bit - 1) % 8
            o, s = (o[0] + ((oc >> 2) & 1), o[1] + ((oc >> 1) & 1), o[2] + (oc & 1)), 1
        else:
            o, s = regions[bit]
        cells.add((smp, 8 * td + o[0], 8 * th + o[1], 8 * tw + o[2], s))
    return cells


def test_pool_matches_dense_maxpool_and_halves_cells():
    rng = np.random.default_rng(21)
    g = O.build(synth.random_occupancy(rng, 2, 2, 4, 2))
    data = rng.standard_normal((g.n_leaves, 3))
    gp, dp = O.pool2_max(g, data)
    assert (gp.gd, gp.gh, gp.gw) == (1, 2, 1)
    dense = torch.from_numpy(O.oc2ten(g, data)).permute(0, 4, 1, 2, 3)
    want = torch.nn.functional.max_pool3d(dense, 2).permute(0, 2, 3, 4, 1).numpy()
    assert np.array_equal(O.oc2ten(gp, dp), want)
    # Each input cell of size >= 2 is halved; every split depth-2 node (a 2^3
    # block of unit voxels) becomes one unit voxel.
    want_cells = set()
    for (smp, d, h, w, s) in _leaf_cells(g):
        if s >= 2:
            want_cells.add((smp, d // 2, h // 2, w // 2, s // 2))
        else:
            want_cells.add((smp, d // 2, h // 2, w // 2, 1))
    assert _leaf_cells(gp) == want_cells
    for t in gp.trees:
        assert O.tree_valid(t) and O.bit(t, 0) == 1


def test_unpool_matches_nearest_upsampling_and_doubles_cells():
    rng = np.random.default_rng(22)
    g = O.build(synth.random_occupancy(rng, 2, 1, 2, 1))
    data = rng.standard_normal((g.n_leaves, 2))
    gu, du = O.unpool2(g, data)
    assert (gu.gd, gu.gh, gu.gw) == (2, 4, 2)
    dense = O.oc2ten(g, data)
    want = dense.repeat(2, axis=1).repeat(2, axis=2).repeat(2, axis=3)
    assert np.array_equal(O.oc2ten(gu, du), want)
    want_cells = set()
    for (smp, d, h, w, s) in _leaf_cells(g):
        if s == 8:
            for o in range(8):
                want_cells.add((smp, 2 * d + 8 * ((o >> 2) & 1), 2 * h + 8 * ((o >> 1) & 1),
                                2 * w + 8 * (o & 1), 8))
        else:
            want_cells.add((smp, 2 * d, 2 * h, 2 * w, 2 * s))
    assert _leaf_cells(gu) == want_cells
    for t in gu.trees:
        assert O.tree_valid(t)


def test_guided_unpool_restores_guide_structure():
    rng = np.random.default_rng(23)
    guide = O.build(synth.random_occupancy(rng, 1, 2, 2, 4))
    x = rng.standard_normal((guide.n_leaves, 2))
    gp, dp = O.pool2_max(guide, x)
    gu, du = O.unpool2(gp, dp, guide=guide)
    assert gu is guide
    want = O.oc2ten(gp, dp).repeat(2, axis=1).repeat(2, axis=2).repeat(2, axis=3)
    assert np.array_equal(O.oc2ten(guide, du), want)
    # plain unpooling of pool(G) is G with its depth-2 splits removed
    plain = O.unpool2_structure(gp)
    for tg, tp in zip(guide.trees, plain.trees):
        bg = O.words_to_bits(tg)
        bg[9:] = 0
        assert np.array_equal(O.words_to_bits(tp), bg)


# ---------------------------------------------------------------------------
# Point clouds (Sec. 5): voxelise, build, per-leaf mean features and votes.
# ---------------------------------------------------------------------------

def test_points_voxelize_floor_and_drop():
    pts = np.array([[0.0, 0.0, 0.0], [7.99, 0.5, 15.999], [8.0, 8.0, 8.0], [-0.01, 1, 1],
                    [16.0, 1, 1], [1, 1, 1]], np.float32)
    batch = np.array([0, 0, 0, 0, 0, 1])
    occ = O.points_voxelize(pts, batch, 1, 2, 1, 2)
    assert occ.shape == (1, 16, 8, 16)
    assert occ.sum() == 2  # the last four are outside the grid or the batch
    assert occ[0, 0, 0, 0] == 1 and occ[0, 7, 0, 15] == 1
    # (8, 8, 8) is outside the 8-voxel-high grid along h
    assert occ[0, 8, :, 8].sum() == 0


def test_points_average_and_vote_by_hand():
    # One empty 8^3 tree with no points but a point block in the corner: the
    # build splits down to that voxel; a second point in the same voxel and
    # a third in a coarse empty leaf far away.
    pts = np.array([[0.5, 0.5, 0.5], [0.25, 0.75, 0.5], [6.5, 6.5, 6.5]], np.float32)
    feat = np.array([[1.0, 10.0], [3.0, 20.0], [5.0, 7.0]], np.float32)
    labels = np.array([2, 1, 4])
    occ = O.points_voxelize(pts, None, 1, 1, 1, 1)
    g = O.build(occ)
    rows = O.points_leaf_rows(g, pts, None)
    assert rows[0] == rows[1] != rows[2]
    avg = O.points_average(g.n_leaves, rows, feat)
    np.testing.assert_allclose(avg[rows[0]], [1.0, 2.0, 15.0])
    np.testing.assert_allclose(avg[rows[2]], [1.0, 5.0, 7.0])
    others = np.setdiff1d(np.arange(g.n_leaves), rows)
    assert np.all(avg[others] == 0)
    vote = O.points_vote(g.n_leaves, rows, labels, 5)
    assert vote[rows[0]] == 1  # tie 1 vs 2: the smaller label
    assert vote[rows[2]] == 4
    assert np.all(vote[others] == -1)


def test_points_leaf_contains_point():
    """Every point's leaf cell contains the point's voxel, for a random cloud."""
    rng = np.random.default_rng(8)
    pts = (rng.random((400, 3)) * np.array([16, 24, 16])).astype(np.float32)
    occ = O.points_voxelize(pts, None, 1, 2, 3, 2)
    g = O.build(occ)
    rows = O.points_leaf_rows(g, pts, None)
    info = O.leaf_info(g)
    def cell(bit):
        # Origin and edge of the cell of bit index `bit` (octant o covers
        # offset ((o>>2)&1, (o>>1)&1, o&1) times the child edge).
        size = 8 if bit == 0 else (4 if bit < 9 else (2 if bit < 73 else 1))
        o, i, edge = np.zeros(3, int), bit, size
        while i > 0:
            oc_ = (i - 1) % 8
            o += np.array([(oc_ >> 2) & 1, (oc_ >> 1) & 1, oc_ & 1]) * edge
            i, edge = (i - 1) // 8, edge * 2
        return o, size

    for p, r in zip(pts, rows):
        t, bit = int(info[r] >> np.uint64(10)), int(info[r] & np.uint64(1023))
        td, th, tw = t // 6, (t // 2) % 3, t % 2
        (d, h, w), s = cell(bit)
        v = np.floor(p).astype(int)
        o = np.array([8 * td + d, 8 * th + h, 8 * tw + w])
        assert np.all(v >= o) and np.all(v < o + s)


# ---------------------------------------------------------------------------
# The supplement's efficient convolution: operation counts.
# ---------------------------------------------------------------------------

def test_truncated_kernel_counts_match_the_paper():
    from paper_1611_05009_amd import reports as R
    # The supplement's figures for an 8^3 cell and a 3^3 kernel.
    assert R.conv_products(8, "naive") == 13824
    assert R.conv_products(8, "truncated") == 3203
    assert round(100.0 * 3203 / 13824, 2) == 23.17


@pytest.mark.parametrize("s", [1, 2, 3, 4, 5, 8])
def test_truncated_kernel_counts_by_enumeration(s):
    """The closed form equals a brute-force count of (voxel, tap) pairs whose
    tap leaves the cell."""
    from paper_1611_05009_amd import reports as R
    n = 0
    for d in range(s):
        for h in range(s):
            for w in range(s):
                for dd in (-1, 0, 1):
                    for dh in (-1, 0, 1):
                        for dw in (-1, 0, 1):
                            q = (d + dd, h + dh, w + dw)
                            n += any(c < 0 or c >= s for c in q)
    assert R.outside_taps(s) == n
