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


def test_mfma_support_query(L):
    # the query is pure host logic
    for cin, cout in [(1, 8), (32, 32), (16, 32), (70, 3)]:
        assert L.oc_conv3x3x3_mfma_supported(cin, cout) in (0, 1)
    # Widths that run in 32-channel blocks: cin a multiple of 32, cout a
    # multiple of 32 up to 256 or a fused width below 32.
    for cin, cout in [(64, 64), (128, 64), (256, 128), (32, 64), (64, 8), (96, 16)]:
        assert L.oc_conv3x3x3_mfma_supported(cin, cout) == 1, (cin, cout)
    for cin, cout in [(64, 130), (48, 32), (64, 3), (32, 288)]:
        assert L.oc_conv3x3x3_mfma_supported(cin, cout) == 0, (cin, cout)
