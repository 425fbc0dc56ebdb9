/* Exported wrappers around the header-only helpers of include/octnet_hip.h,
 * compiled by tests/test_header_helpers.py with a plain C compiler (gcc
 * -std=c99) into a small shared library that the test loads with ctypes.
 * Compiling this file is itself the check that the header is valid C. */
#include "octnet_hip.h"

int hh_parent(int i) { return oc_parent(i); }
int hh_child(int i) { return oc_child(i); }
int hh_bit(const uint32_t* t, int i) { return oc_bit(t, i); }
int hh_data_idx(const uint32_t* t, int i) { return oc_data_idx(t, i); }
int hh_n_leaves(const uint32_t* t) { return oc_n_leaves(t); }
int hh_leaf_at(const uint32_t* t, int d, int h, int w, int* depth) { return oc_leaf_at(t, d, h, w, depth); }
int hh_canonical(const uint32_t* t) { return oc_tree_canonical(t); }
int hh_validate(const uint32_t* trees, int64_t n) { return oc_validate_host(trees, n); }
