"""The header-only helpers of include/octnet_hip.h (oc_parent, oc_child,
oc_bit, oc_data_idx, oc_n_leaves, oc_leaf_at, oc_tree_canonical,
oc_validate_host), compiled from tests/header_helpers.c by a plain C
compiler, checked against what pins them:

- Eq. 1-2: the closed forms, exhaustively;
- the Fig. 3 split string: its set bits and 50 leaves;
- Eq. 3: the oracle's data index (its Eq. 3 and its breadth-first rank by
  enumeration, both pinned by the supplement's worked example) for every leaf
  of random canonical trees;
- voxel addressing (Sec. 3.2): the oracle's row map of one tree;
- canonical form: the oracle's check on trees with orphan bits.

The supplement's worked example is a quadtree (branching 4); the header's
helpers are the octree form (branching 8), so that example pins them only
through the oracle's Eq. 3, which it checks at both branching factors.
"""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

import octref as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")


@pytest.fixture(scope="module")
def H(tmp_path_factory):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    out = str(tmp_path_factory.mktemp("hh") / "libhh.so")
    subprocess.check_call([cc, "-std=c99", "-Wall", "-Werror", "-O1", "-fPIC", "-shared",
                           "-I", os.path.join(ROOT, "include"), "-o", out,
                           os.path.join(HERE, "header_helpers.c")])
    L = ctypes.CDLL(out)
    P, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    for name, args in [("hh_parent", [i32]), ("hh_child", [i32]), ("hh_bit", [P, i32]),
                       ("hh_data_idx", [P, i32]), ("hh_n_leaves", [P]),
                       ("hh_leaf_at", [P, i32, i32, i32, P]), ("hh_canonical", [P]),
                       ("hh_validate", [P, i64])]:
        f = getattr(L, name)
        f.restype = i32
        f.argtypes = args
    return L


def test_header_compiles_as_cplusplus(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("no C++ compiler")
    src = tmp_path / "x.cpp"
    src.write_text('#include "octnet_hip.h"\nint main() { const uint32_t t[4] = {1, 0, 0, 0};'
                   ' return oc_n_leaves(t) == 8 ? 0 : 1; }\n')
    exe = str(tmp_path / "x")
    subprocess.check_call([cxx, "-std=c++17", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                           "-o", exe, str(src)])
    assert subprocess.call([exe]) == 0


def _words(bits):
    return np.ascontiguousarray(O.bits_to_words(bits), dtype=np.uint32)


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def _read_golden(name):
    vals = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if line and not line.startswith("#"):
            k, v = [x.strip() for x in line.split("=", 1)]
            vals[k] = v
    return vals


def _random_bits(rng, p0=0.9, p1=0.5, p2=0.4):
    bits = np.zeros(73, dtype=np.uint8)
    if rng.random() < p0:
        bits[0] = 1
        for o in range(8):
            if rng.random() < p1:
                bits[1 + o] = 1
                for q in range(8):
                    bits[9 + 8 * o + q] = rng.random() < p2
    return bits


def test_parent_child_closed_forms(H):
    assert H.hh_parent(0) == -1
    for i in range(1, 585):
        p = H.hh_parent(i)
        assert p == (i - 1) // 8 and H.hh_child(p) <= i < H.hh_child(p) + 8
    for i in range(73):
        assert H.hh_child(i) == 8 * i + 1


def test_fig3_string(H):
    g = _read_golden("fig3_octree_bits.txt")
    s = np.array([int(c) for c in g["bits"].replace(" ", "")], dtype=np.uint8)
    bits = np.zeros(73, dtype=np.uint8)
    bits[:len(s)] = s
    w = _words(bits)
    assert [i for i in range(73) if H.hh_bit(_ptr(w), i)] == [int(x) for x in g["split_bits"].split()]
    assert H.hh_n_leaves(_ptr(w)) == int(g["n_leaves"])
    assert H.hh_canonical(_ptr(w)) == 1
    # Eq. 3 ranks the 50 leaves 0..49 in ascending bit order.
    leaves = [i for i in range(585) if O.data_idx_bfs(bits, 8, 3, i) >= 0]
    assert [H.hh_data_idx(_ptr(w), i) for i in leaves] == list(range(int(g["n_leaves"])))


def test_data_idx_matches_oracle_on_random_trees(H):
    rng = np.random.default_rng(11)
    for _ in range(120):
        bits = _random_bits(rng)
        w = _words(bits)
        assert H.hh_n_leaves(_ptr(w)) == O.tree_n_leaves(w)
        for i in range(585):
            r = O.data_idx_bfs(bits, 8, 3, i)
            if r >= 0:
                assert H.hh_data_idx(_ptr(w), i) == r == O.data_idx_eq3(bits, 8, i), i
        for i in range(-3, 80):
            assert H.hh_bit(_ptr(w), i) == (int(bits[i]) if 0 <= i < 73 else 0)


def test_leaf_at_matches_oracle_rowmap(H):
    rng = np.random.default_rng(12)
    depth = ctypes.c_int(-1)
    for _ in range(40):
        bits = _random_bits(rng)
        w = _words(bits)
        g = O.make_grid(w[None, :], 1, 1, 1, 1)
        rm = O.rowmap(g)[0]
        info = O.leaf_info(g)
        for d in range(8):
            for h in range(8):
                for x in range(8):
                    i = H.hh_leaf_at(_ptr(w), d, h, x, ctypes.byref(depth))
                    # the oracle's leaf at this voxel, as (bit index) of its row
                    assert i == int(info[rm[d, h, x]] & np.uint64(1023))
                    assert H.hh_data_idx(_ptr(w), i) == rm[d, h, x]
                    assert depth.value == (0 if i == 0 else 1 if i < 9 else 2 if i < 73 else 3)
    assert H.hh_leaf_at(_ptr(w), 8, 0, 0, None) == -1


def test_canonical_and_validate_host_match_oracle(H):
    rng = np.random.default_rng(13)
    trees = []
    for k in range(200):
        bits = _random_bits(rng)
        w = _words(bits)
        if k % 3 == 1:
            w[rng.integers(0, 3)] ^= np.uint32(1) << np.uint32(rng.integers(0, 32))  # may orphan a bit
        if k % 17 == 5:
            w[3] = np.uint32(1)  # beyond the 73-bit string
        assert H.hh_canonical(_ptr(w)) == int(O.tree_valid(w)), (k, w)
        trees.append(w)
    good = np.ascontiguousarray([t for t in trees if O.tree_valid(t)], dtype=np.uint32)
    allt = np.ascontiguousarray(trees, dtype=np.uint32)
    assert H.hh_validate(_ptr(good), len(good)) == 0
    assert H.hh_validate(_ptr(allt), len(allt)) == -2
    assert H.hh_validate(None, 3) == -1
