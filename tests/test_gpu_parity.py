"""GPU parity: every C-ABI operation against the CPU oracle.

Structure, prefix, leaf index and row maps must match bit for bit; copies and
maxima (pool, unpool, oc2ten) exactly; convolution features within
|gpu - oracle| <= 1e-5 + 1e-4 |oracle| in fp32.
"""
import numpy as np
import pytest
import torch

import octref as O
from common import assert_close, log, trees_np, workload_occupancy
from paper_1611_05009_amd import synth

pytestmark = pytest.mark.gpu

oc = None


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    global oc
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1611_05009_amd import octnet
    octnet.lib()  # raises if the HIP library is missing
    oc = octnet
    torch.cuda.set_device(0)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.detach().cpu().numpy()


# Tiny grids: several trees per axis, odd extents, two samples.
SMALL = [
    (1, 1, 1, 1, 1),
    (2, 2, 3, 2, 2),
    (3, 1, 2, 5, 3),
    (4, 2, 2, 2, 4),
]


def small_occ(seed, n, gd, gh, gw):
    return synth.random_occupancy(np.random.default_rng(seed), n, gd, gh, gw)


def check_structure(g, ref):
    assert g.dims() == (ref.n, ref.gd, ref.gh, ref.gw)
    assert np.array_equal(trees_np(g.trees), ref.trees)
    assert np.array_equal(host(g.prefix), ref.prefix)
    assert g.n_leaves == ref.n_leaves


# ----------------------------------------------------------------------------
# Structure
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("rule", ["mixed", "any"])
@pytest.mark.parametrize("case", SMALL)
def test_build_index_rowmap_bitexact(case, rule):
    occ = small_occ(*case)
    ref = O.build(occ, rule)
    g = oc.build(dev(occ), rule)
    check_structure(g, ref)
    assert np.array_equal(host(oc.leaf_index(g)).view(np.uint64), O.leaf_info(ref))
    assert np.array_equal(host(oc.rowmap(g)), O.rowmap(ref))
    assert oc.validate(g) == 0
    g2 = oc.from_trees(g.trees.clone(), *g.dims())
    assert np.array_equal(host(g2.prefix), ref.prefix)


@pytest.mark.parametrize("case", [(6, 1, 1, 1, 37), (7, 2, 1, 2, 70), (8, 1, 2, 1, 64)])
def test_build_wide_grids(case):
    """Grid widths past one build workgroup's 32 trees: odd (8-byte row
    pieces), even with a partial last workgroup, and whole workgroups."""
    occ = small_occ(*case)
    for rule in ("mixed", "any"):
        ref = O.build(occ, rule)
        g = oc.build(dev(occ), rule)
        check_structure(g, ref)


@pytest.mark.parametrize("fill", ["empty", "full", "checker"])
def test_build_degenerate_grids(fill):
    occ = np.zeros((2, 16, 8, 24), dtype=np.uint8)
    if fill == "full":
        occ[:] = 1
    elif fill == "checker":
        occ[:] = (np.indices(occ.shape[1:]).sum(0) % 2)[None]
    for rule in ("mixed", "any"):
        ref = O.build(occ, rule)
        g = oc.build(dev(occ), rule)
        check_structure(g, ref)
        assert np.array_equal(host(oc.leaf_index(g)).view(np.uint64), O.leaf_info(ref))


@pytest.mark.parametrize("nt", [1, 15, 16, 17, 4095, 4096, 4097, 65537, (1 << 20) + 3])
def test_prefix_across_scan_chunks(nt):
    """oc_prefix (Eq. 3's per-tree offsets: an exclusive scan of 1 + 7 x set
    bits) for tree counts around the scan's per-thread (16 trees) and
    per-block (4096 trees) chunks, into an aligned and a misaligned output
    (the scan's vector and element paths), against the oracle's prefix."""
    import ctypes
    words = synth.random_trees(np.random.default_rng(nt), nt, 1, 1, 1)
    ref = O.prefix_of(words)
    log("prefix nt=%d" % nt)
    g = oc.from_trees(dev(words.view(np.int32)), nt, 1, 1, 1)
    assert g.n_leaves == ref[-1]
    assert np.array_equal(host(g.prefix), ref)
    buf = torch.empty(nt + 2, dtype=torch.int64, device="cuda")
    out = buf[1:]  # 8-byte aligned, not 16
    ws = oc.structure_workspace(nt)
    nl = ctypes.c_int64(0)
    rc = oc.lib().oc_prefix(oc._ptr(g.trees), nt, oc._ptr(out), ctypes.byref(nl), oc._ptr(ws), ws.numel(),
                            oc._stream())
    assert rc == 0 and nl.value == ref[-1]
    assert np.array_equal(host(out), ref)


def test_validate_flags_noncanonical_trees():
    occ = small_occ(5, 1, 2, 2, 2)
    g = oc.build(dev(occ))
    t = trees_np(g.trees).copy()
    t[0] = [0, 0, 0, 0]
    t[0][0] = 1 << 9     # depth-2 bit under an unsplit root
    t[1][2] |= 1 << 12   # bit 76: beyond the 73-bit string
    # oc_prefix, where trees made elsewhere enter, rejects them...
    with pytest.raises(oc.OctNetError, match="non-canonical"):
        oc.from_trees(dev(t.view(np.int32)), *g.dims())
    # ...and oc_validate counts them (it needs no prefix).
    bad = oc.Octree(*g.dims(), dev(t.view(np.int32)), g.prefix, g.n_leaves)
    assert oc.validate(bad) == 2
    # The host form agrees tree by tree (header-only oc_validate_host is
    # pinned against the oracle in test_header_helpers.py).
    assert [O.tree_valid(w) for w in t[:3]] == [False, False, True]


@pytest.mark.parametrize("key", ["c1", "c2", "c3", "c4", "c5"])
def test_workload_structure_bitexact(key):
    log("structure %s" % key)
    occ, _ = workload_occupancy(key)
    ref = O.build(occ)
    g = oc.build(dev(occ))
    check_structure(g, ref)
    info = host(oc.leaf_index(g)).view(np.uint64)
    assert np.array_equal(info, O.leaf_info(ref))


# ----------------------------------------------------------------------------
# oc2ten / ten2oc
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("case", SMALL)
def test_oc2ten_ten2oc(case):
    occ = small_occ(*case)
    ref = O.build(occ)
    g = oc.build(dev(occ))
    rng = np.random.default_rng(77)
    data = rng.standard_normal((ref.n_leaves, 3)).astype(np.float32)
    dense = host(oc.oc2ten(g, dev(data)))
    assert np.array_equal(dense, O.oc2ten(ref, data).astype(np.float32))
    x = rng.standard_normal(ref.dense_shape + (5,)).astype(np.float32)
    assert_close(host(oc.ten2oc(g, dev(x), "avg")), O.ten2oc(ref, x, "avg"), "ten2oc avg")
    assert np.array_equal(host(oc.ten2oc(g, dev(x), "max")), O.ten2oc(ref, x, "max").astype(np.float32))


@pytest.mark.parametrize("c", [1, 4, 8, 6])
def test_ten2oc_channel_widths(c):
    """ten2oc over 4-channel chunks: whole 16-byte chunks (c = 4, 8), a
    partial last chunk (6) and one channel; both split rules' structures."""
    rng = np.random.default_rng(100 + c)
    occ = synth.random_occupancy(rng, 2, 2, 3, 2)
    for rule in ("mixed", "any"):
        ref = O.build(occ, rule)
        g = oc.build(dev(occ), rule)
        x = rng.standard_normal(ref.dense_shape + (c,)).astype(np.float32)
        assert_close(host(oc.ten2oc(g, dev(x), "avg")), O.ten2oc(ref, x, "avg"), "ten2oc avg c=%d" % c)
        assert np.array_equal(host(oc.ten2oc(g, dev(x), "max")), O.ten2oc(ref, x, "max").astype(np.float32))


# ----------------------------------------------------------------------------
# Convolution
# ----------------------------------------------------------------------------

CHANNELS = [(1, 8), (3, 5), (4, 16), (8, 16), (16, 32), (32, 32), (32, 8), (70, 3), (16, 4), (32, 1), (8, 2), (4, 3)]


def conv_case(seed, cin, cout, shape=(2, 3, 2, 3)):
    rng = np.random.default_rng(seed)
    occ = synth.random_occupancy(rng, *shape)
    ref = O.build(occ)
    x = rng.standard_normal((ref.n_leaves, cin)).astype(np.float32)
    w = (rng.standard_normal((cout, cin, 3, 3, 3)) / np.sqrt(27 * cin)).astype(np.float32)
    b = rng.standard_normal(cout).astype(np.float32)
    return occ, ref, x, w, b


@pytest.mark.parametrize("impl", ["generic", "mfma", "gemm", "truncated"])
@pytest.mark.parametrize("cin,cout", CHANNELS)
def test_conv_small(cin, cout, impl):
    if impl == "mfma" and not oc.mfma_supported(cin, cout):
        pytest.skip("no MFMA kernel for (%d, %d)" % (cin, cout))
    occ, ref, x, w, b = conv_case(1000 + cin * 7 + cout, cin, cout)
    g = oc.build(dev(occ))
    want = O.conv3(ref, x, w, b)
    got = host(oc.conv3x3x3(g, dev(x), dev(w), dev(b), impl=impl))
    # Every implementation, the truncated-kernel one included (its
    # differences x_nb - x_l cancel against the constant part, yet it stays
    # within the element-wise bar), at 1e-5 + 1e-4 |oracle|.
    assert_close(got, want, "conv %s %dx%d" % (impl, cin, cout))
    got_r = host(oc.conv3x3x3(g, dev(x), dev(w), None, relu=True, impl=impl))
    assert_close(got_r, np.maximum(O.conv3(ref, x, w, None), 0), "conv relu")


@pytest.mark.parametrize("impl", ["generic", "mfma", "gemm", "truncated"])
def test_conv_degenerate_structures(impl):
    cin, cout = 32, 32
    if impl == "mfma" and not oc.mfma_supported(cin, cout):
        pytest.skip("no MFMA kernel")
    rng = np.random.default_rng(31)
    cases = {
        "single_tree_empty": np.zeros((1, 8, 8, 8), np.uint8),
        "all_split": None,
        "one_voxel": np.zeros((1, 8, 16, 8), np.uint8),
    }
    cases["one_voxel"][0, 7, 8, 0] = 1
    for name, occ in cases.items():
        if occ is None:
            occ = np.ones((1, 16, 8, 8), np.uint8)
            ref = O.build(occ, "any")
            g = oc.build(dev(occ), "any")
        else:
            ref = O.build(occ)
            g = oc.build(dev(occ))
        x = rng.standard_normal((ref.n_leaves, cin)).astype(np.float32)
        w = (rng.standard_normal((cout, cin, 3, 3, 3)) / np.sqrt(27 * cin)).astype(np.float32)
        got = host(oc.conv3x3x3(g, dev(x), dev(w), impl=impl))
        assert_close(got, O.conv3(ref, x, w), "conv %s %s" % (impl, name))


@pytest.mark.parametrize("impl", ["auto", "mfma", "gemm"])
@pytest.mark.parametrize("cin,cout", [(64, 64), (128, 64), (256, 128), (64, 130), (32, 64), (64, 8),
                                      (96, 16), (64, 32), (64, 3)])
def test_conv_wide_channels(cin, cout, impl):
    """Widths of the encoder-decoder's coarse levels, which have no fused
    variant: the window-sum GEMM path, and the fused kernels run in 32-channel
    blocks ("mfma"; auto takes it on large structures only)."""
    if impl == "mfma" and not oc.mfma_supported(cin, cout):
        pytest.skip("no channel blocks for (%d, %d)" % (cin, cout))
    occ, ref, x, w, b = conv_case(5000 + cin + cout, cin, cout, shape=(2, 2, 3, 2))
    g = oc.build(dev(occ))
    want = O.conv3(ref, x, w, b)
    got = host(oc.conv3x3x3(g, dev(x), dev(w), dev(b), impl=impl))
    assert_close(got, want, "conv %s %dx%d" % (impl, cin, cout))
    got_r = host(oc.conv3x3x3(g, dev(x), dev(w), None, relu=True, impl=impl))
    assert_close(got_r, np.maximum(O.conv3(ref, x, w, None), 0), "conv %s relu %dx%d" % (impl, cin, cout))


def test_conv_closed_form_single_cell():
    g = oc.build(dev(np.zeros((1, 8, 8, 8), np.uint8)))
    y = host(oc.conv3x3x3(g, dev(np.ones((1, 1), np.float32)), dev(np.ones((1, 1, 3, 3, 3), np.float32))))
    assert abs(float(y[0, 0]) - 20.796875) <= 1e-5


def test_conv_deterministic():
    occ, ref, x, w, b = conv_case(4242, 32, 32)
    g = oc.build(dev(occ))
    a = host(oc.conv3x3x3(g, dev(x), dev(w), dev(b)))
    c = host(oc.conv3x3x3(g, dev(x), dev(w), dev(b)))
    assert np.array_equal(a, c)


# ----------------------------------------------------------------------------
# Pool / unpool
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("case", [(7, 1, 2, 2, 2), (8, 2, 4, 2, 6), (9, 3, 2, 4, 2)])
def test_pool_unpool_small(case):
    occ = small_occ(*case)
    ref = O.build(occ)
    g = oc.build(dev(occ))
    rng = np.random.default_rng(5)
    x = rng.standard_normal((ref.n_leaves, 6)).astype(np.float32)
    rp, rdp = O.pool2_max(ref, x)
    gp, dp = oc.pool2(g, dev(x))
    check_structure(gp, rp)
    assert np.array_equal(host(dp), rdp.astype(np.float32))
    # plain unpooling of the pooled grid
    ru, rdu = O.unpool2(rp, rdp.astype(np.float32))
    gu, du = oc.unpool2(gp, dp)
    check_structure(gu, ru)
    assert np.array_equal(host(du), rdu.astype(np.float32))
    # guided unpooling back onto the input structure
    rg, rdg = O.unpool2(rp, rdp.astype(np.float32), guide=ref)
    gg, dg = oc.unpool2(gp, dp, guide=g)
    check_structure(gg, rg)
    assert np.array_equal(host(dg), rdg.astype(np.float32))


def test_pool_rejects_odd_grid_and_guided_mismatch():
    occ = small_occ(3, 1, 2, 2, 2)
    g = oc.build(dev(occ))
    g_odd = oc.build(dev(small_occ(3, 1, 3, 2, 2)))
    with pytest.raises(oc.OctNetError, match="invalid argument"):
        oc.pool2_structure(g_odd)
    gp, _ = oc.pool2(g, dev(np.zeros((g.n_leaves, 1), np.float32)))
    other = oc.build(dev(small_occ(4, 1, 2, 2, 2)))
    with pytest.raises(oc.OctNetError, match="structure"):
        oc.unpool2_structure(gp, guide=other)


def test_plain_unpool_of_unsplit_roots():
    occ = np.zeros((1, 8, 16, 8), np.uint8)
    occ[0, 1, 9, 3] = 1
    ref = O.build(occ)
    g = oc.build(dev(occ))
    x = np.arange(ref.n_leaves * 2, dtype=np.float32).reshape(-1, 2)
    ru, rdu = O.unpool2(ref, x)
    gu, du = oc.unpool2(g, dev(x))
    check_structure(gu, ru)
    assert np.array_equal(host(du), rdu.astype(np.float32))


def test_relu():
    x = torch.randn(1001, device="cuda")
    y = x.clone()
    oc.relu_(y)
    assert torch.equal(y, torch.clamp(x, min=0))
    z = x.clone()
    oc.relu_(z[1:])  # a view 4 bytes past a 16-byte boundary
    assert torch.equal(z[1:], torch.clamp(x[1:], min=0)) and z[0] == x[0]
