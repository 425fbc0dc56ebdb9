"""Host-side checks of the C ABI: the library loads, exports every function
include/octnet_hip.h declares, and rejects bad arguments before any launch
(no GPU work is issued by these calls)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "octnet_hip.h")


def _header_text():
    return re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)


def inline_helpers():
    """Header-only helpers (static inline, not exported by the library)."""
    return sorted(set(re.findall(r"OC_INLINE\s+\w+\s+(oc_\w+)\s*\(", _header_text())))


def declared_functions():
    """Functions the library exports: every oc_* the header names, minus the
    header-only helpers."""
    names = set(re.findall(r"\b(oc_\w+)\s*\(", _header_text()))
    return sorted(names - set(inline_helpers()))


@pytest.fixture(scope="module")
def L():
    from paper_1611_05009_amd import octnet
    if not os.path.exists(octnet.LIB_PATH):
        from paper_1611_05009_amd import build_lib
        build_lib.build()
    return octnet.lib()


def test_header_declares_the_binding_surface():
    from paper_1611_05009_amd import octnet
    assert declared_functions() == sorted(octnet.SIGNATURES)


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_header_only_helpers_are_present():
    assert inline_helpers() == sorted([
        "oc_parent", "oc_child", "oc_bit", "oc_popc_below", "oc_data_idx", "oc_n_leaves",
        "oc_leaf_at", "oc_tree_canonical", "oc_validate_host"])


def test_error_strings_and_version(L):
    assert L.oc_version() >= 100
    for code, word in [(0, b"ok"), (-1, b"invalid"), (-2, b"structure"), (-3, b"workspace"),
                       (-4, b"HIP"), (-5, b"overflow")]:
        assert word in L.oc_error_string(code)


def test_null_pointers_and_bad_sizes_are_rejected_on_the_host(L):
    nl = ctypes.c_int64(0)
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: checks fail first
    assert L.oc_build(None, 1, 1, 1, 1, 0, fake, fake, ctypes.byref(nl), fake, 1 << 20, None) == -1
    assert L.oc_build(fake, 0, 1, 1, 1, 0, fake, fake, ctypes.byref(nl), fake, 1 << 20, None) == -1
    assert L.oc_build(fake, 1, 1, 1, 1, 7, fake, fake, ctypes.byref(nl), fake, 1 << 20, None) == -1
    assert L.oc_build(fake, 1, 1, 1, 1, 0, fake, fake, ctypes.byref(nl), fake, 16, None) == -3
    assert b"workspace" in L.oc_last_error()
    # odd tree grid for pooling
    assert L.oc_pool2_structure(fake, 1, 3, 2, 2, fake, fake, ctypes.byref(nl), fake, 1 << 20, None) == -1
    # channel limits, leaf count limits, workspace size
    nb = ctypes.c_size_t(0)
    assert L.oc_conv3x3x3_workspace(8, 100, 32, 32, ctypes.byref(nb)) == 0 and nb.value > 0
    args = [fake, fake, 1, 2, 2, 2]
    assert L.oc_conv3x3x3(*args, 100, fake, 0, fake, None, 8, 0, fake, fake, nb.value, None) == -1
    assert L.oc_conv3x3x3(*args, 100, fake, 300, fake, None, 8, 0, fake, fake, nb.value, None) == -1
    assert L.oc_conv3x3x3(*args, 1 << 31, fake, 4, fake, None, 8, 0, fake, fake, nb.value, None) == -5
    assert L.oc_conv3x3x3(*args, 5000, fake, 4, fake, None, 8, 0, fake, fake, nb.value, None) == -1
    assert L.oc_conv3x3x3(*args, 100, fake, 32, fake, None, 32, 0, fake, fake, 64, None) == -3
    assert L.oc_conv3x3x3_ex(*args, 100, fake, 32, fake, None, 32, 0, fake, fake, nb.value, 9, None) == -1
    assert L.oc_relu(None, 10, None) == -1
    assert L.oc_relu(fake, -1, None) == -1


def test_workspace_by_slot_count(L):
    """The exact-size query adds the slot-sized parts (boundary sums, 6^3
    node tables, set masks) per slot to the fixed parts; the size-only query
    is the one for the bound (n_leaves - n_trees) / 7 slots."""
    fake = ctypes.c_void_p(0x1000)
    for nt, nl, cin, cout in [(8, 100, 32, 32), (4096, 300000, 16, 32), (64, 4000, 8, 16), (64, 4000, 1, 8),
                              (512, 60000, 64, 64)]:
        nb, one, two, big = (ctypes.c_size_t(0) for _ in range(4))
        assert L.oc_conv3x3x3_workspace(nt, nl, cin, cout, ctypes.byref(nb)) == 0
        bound = max(1, (nl - nt) // 7) if nl > nt + 7 else 1
        assert L.oc_conv3x3x3_workspace_slots(nt, nl, cin, cout, bound, ctypes.byref(big)) == 0
        assert big.value == nb.value, (nt, nl, cin, cout)
        assert L.oc_conv3x3x3_workspace_slots(nt, nl, cin, cout, 10 * bound, ctypes.byref(big)) == 0
        assert big.value == nb.value
        assert L.oc_conv3x3x3_workspace_slots(nt, nl, cin, cout, 0, ctypes.byref(one)) == 0
        assert L.oc_conv3x3x3_workspace_slots(nt, nl, cin, cout, 1, ctypes.byref(two)) == 0
        assert one.value == two.value <= nb.value
        fused = L.oc_conv3x3x3_mfma_supported(cin, cout) == 1 and (cin <= 32)
        if fused and bound > 3000:
            # 26 cin floats + a 216-entry table + a mask word per slot
            assert L.oc_conv3x3x3_workspace_slots(nt, nl, cin, cout, 3001, ctypes.byref(big)) == 0
            per = (big.value - one.value) / 3000
            assert abs(per - (26 * cin * 4 + 216 * 4 + 4)) < 1, per
        # the capacity a workspace holds round-trips the size by slot count
        cap = ctypes.c_int64(-7)
        for k in sorted({1, 2, 3, 5, 17, 255, 256, 257, bound // 3, bound - 1, bound}):
            if k < 1:
                continue
            assert L.oc_conv3x3x3_workspace_slots(nt, nl, cin, cout, k, ctypes.byref(big)) == 0
            assert L.oc_conv3x3x3_workspace_capacity(nt, nl, cin, cout, big.value, ctypes.byref(cap)) == 0
            want = min(k, bound) if fused or L.oc_conv3x3x3_mfma_supported(cin, cout) == 1 else 0
            assert cap.value == want, (nt, nl, cin, cout, k, cap.value)
            if want > 1:  # one byte less holds one slot less
                assert L.oc_conv3x3x3_workspace_capacity(nt, nl, cin, cout, big.value - 1,
                                                          ctypes.byref(cap)) == 0
                assert cap.value == want - 1, (nt, nl, cin, cout, k, cap.value)
        assert L.oc_conv3x3x3_workspace_capacity(nt, nl, cin, cout, one.value - 1, ctypes.byref(cap)) == -3
        # below the one-slot size the convolution refuses the workspace
        args = [fake, fake, 1, 2, 2, 2] if nt == 8 else None
        if args:
            assert L.oc_conv3x3x3(*args, nl, fake, cin, fake, None, cout, 0, fake, fake, one.value - 1,
                                  None) == -3


def test_mfma_support_query(L):
    # the query is pure host logic
    for cin, cout in [(1, 8), (32, 32), (16, 32), (70, 3)]:
        assert L.oc_conv3x3x3_mfma_supported(cin, cout) in (0, 1)
    # Widths that run in 32-channel blocks: cin a multiple of 32, cout a
    # multiple of 32 up to 256 or a fused width below 32.
    for cin, cout in [(64, 64), (128, 64), (256, 128), (32, 64), (64, 8), (96, 16), (64, 3)]:
        assert L.oc_conv3x3x3_mfma_supported(cin, cout) == 1, (cin, cout)
    for cin, cout in [(64, 130), (48, 32), (32, 288), (64, 40)]:
        assert L.oc_conv3x3x3_mfma_supported(cin, cout) == 0, (cin, cout)
