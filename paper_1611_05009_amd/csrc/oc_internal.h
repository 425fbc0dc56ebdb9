// Internal declarations shared by the library's translation units.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "oc_device.h"

namespace oci {

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Prefix scan of int32 counts (n entries) into int64 prefix (n + 1 entries).
// The workspace starts with the counts buffer (scan_counts_buffer).
size_t scan_workspace(int64_t n);
int32_t* scan_counts_buffer(void* ws);
hipError_t scan_counts(const int32_t* counts, int64_t n, int64_t* prefix, void* ws, hipStream_t s);
// k (<= kMaxScans) scans of length n in three launches: ws[i] is a scan
// workspace whose counts buffer holds the counts, prefix[i] the output.
constexpr int kMaxScans = 8;
hipError_t scan_counts_set(int k, void* const* ws, int64_t n, int64_t* const* prefix, hipStream_t s);

hipError_t launch_build(const uint8_t* occ, int n, int gd, int gh, int gw, int rule,
                        uint32_t* trees, int32_t* counts, hipStream_t s);
hipError_t launch_count(const uint32_t* trees, int64_t nt, int32_t* counts, hipStream_t s);
hipError_t launch_validate(const uint32_t* trees, int64_t nt, int32_t* bad, hipStream_t s);
hipError_t launch_leaf_index(const uint32_t* trees, const int64_t* prefix, int64_t nt,
                             uint64_t* info, hipStream_t s);
hipError_t launch_rowmap(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
                         int gw, int64_t* rowmap, hipStream_t s);
hipError_t launch_pool_structure(const uint32_t* in, int n, int gd, int gh, int gw, uint32_t* out,
                                 int32_t* counts, hipStream_t s);
hipError_t launch_unpool_structure(const uint32_t* in, const uint32_t* guide, int n, int gd, int gh,
                                   int gw, uint32_t* out, int32_t* counts, int32_t* mismatch,
                                   hipStream_t s);

hipError_t launch_oc2ten(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
                         int gw, const float* data, int c, float* dense, hipStream_t s);
hipError_t launch_ten2oc(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
                         int gw, const float* dense, int c, int pool, float* data, hipStream_t s);
hipError_t launch_pool_max(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd,
                           int gh, int gw, const float* in, int c, const uint32_t* out_trees,
                           const int64_t* out_prefix, float* out, hipStream_t s);
hipError_t launch_unpool(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh,
                         int gw, const float* in, int c, const uint32_t* out_trees,
                         const int64_t* out_prefix, float* out, hipStream_t s);
hipError_t launch_relu(float* x, int64_t count, hipStream_t s);
// Gradients (the arguments mirror the forward calls; dy/din are the output
// and input gradients).  Every din row is written (no clearing needed).
hipError_t launch_pool_max_bwd(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd,
                               int gh, int gw, const float* in, int c, const uint32_t* out_trees,
                               const int64_t* out_prefix, const float* dy, float* din,
                               hipStream_t s);
hipError_t launch_unpool_bwd(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd,
                             int gh, int gw, int64_t in_n_leaves, int c, const uint32_t* out_trees,
                             const int64_t* out_prefix, const float* dy, float* din,
                             hipStream_t s);
hipError_t launch_relu_bwd(const float* y, const float* dy, float* din, int64_t count,
                           hipStream_t s);
// Channel concatenation of two leaf arrays and its gradient (da, db may be null).
hipError_t launch_concat(const float* a, int ca, const float* b, int cb, int64_t n_rows, float* out,
                         hipStream_t s);
hipError_t launch_split(const float* dout, int ca, int cb, int64_t n_rows, float* da, float* db,
                        hipStream_t s);
// Point clouds: voxelise (clears occ first), the leaf row of each point,
// per-leaf feature means (out [n_leaves][c + 1]; count: n_leaves words of
// scratch) and label majority votes (hist: n_leaves * L words of scratch).
hipError_t launch_voxelize(const float* pts, const int32_t* batch, int64_t n_pts, int n, int gd, int gh,
                           int gw, uint8_t* occ, hipStream_t s);
hipError_t launch_point_rows(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                             const float* pts, const int32_t* batch, int64_t n_pts, int32_t* rows,
                             hipStream_t s);
hipError_t launch_point_means(const int32_t* rows, int64_t n_pts, const float* feat, int c,
                              int64_t n_leaves, float* out, uint32_t* count, hipStream_t s);
hipError_t launch_label_vote(const int32_t* rows, int64_t n_pts, const int32_t* labels, int L,
                             int64_t n_leaves, int32_t* out, uint32_t* hist, hipStream_t s);
// out = a + b (out may alias a or b).
hipError_t launch_add(const float* a, const float* b, float* out, int64_t count, hipStream_t s);

// Convolution.
struct ConvArgs {
  const uint32_t* trees;
  const int64_t* prefix;
  int n, gd, gh, gw;
  int64_t n_trees, n_leaves;
  const float* in;
  int cin;
  const float* weight;
  const float* bias;
  int cout;
  int relu;
  float* out;
  // Internal: the fused kernels write each cell's sum (|l| times Eq. 8's
  // mean) instead of its mean; only where conv_runs_fused holds.
  int sum_cells = 0;
  // Boundary-sum slots the workspace holds (conv_slot_capacity); -1: the
  // size-only bound.
  int64_t slot_cap = -1;
};
// Workspace bound for every canonical structure of this size.
size_t conv_workspace(int64_t n_trees, int64_t n_leaves, int cin, int cout);
// Workspace for a structure with `slots` split trees plus split depth-1
// nodes (at least 1).
size_t conv_workspace_slots(int64_t n_trees, int64_t n_leaves, int cin, int cout, int64_t slots);
// Slots a workspace of ws_bytes holds (at most the bound; 0 where the
// layer has no fused variant); -1 below the one-slot size.
int64_t conv_slot_capacity(int64_t n_trees, int64_t n_leaves, int cin, int cout, size_t ws_bytes);
// *count = split trees plus split depth-1 nodes (asynchronous on s).
hipError_t launch_count_slots(const uint32_t* trees, int64_t n_trees, unsigned long long* count,
                              hipStream_t s);
bool conv_mfma_supported(int cin, int cout);
// The implementation OC_CONV_AUTO runs: 2 (fused MFMA kernels, in channel
// blocks for wide layers on large structures) or 3 (window-sum GEMM).
int conv_auto_impl(int64_t n_leaves, int cin, int cout);
// Whether launch_conv_execute with impl runs the fused MFMA kernels (directly
// or in channel blocks) for these arguments.
bool conv_runs_fused(const ConvArgs& a, int impl);
// Structure- and weight-dependent preparation into the workspace (the
// weight pointer of `a` is read, the features are not).
hipError_t launch_conv_prepare(const ConvArgs& a, void* ws, hipStream_t s);
// The convolution proper; impl: 1 generic, 2 mfma (caller checked support),
// 3 window-sum GEMM.
hipError_t launch_conv_execute(const ConvArgs& a, void* ws, int impl, hipStream_t s);
// The paper's efficient convolution (constant part plus truncated kernels
// at boundary voxels), VALU; info: n_leaves words of scratch.
hipError_t launch_conv_truncated(const ConvArgs& a, uint64_t* info, hipStream_t s);
// Bytes of the window-sum buffer of the GEMM path (one row chunk).
size_t conv_gemm_buffer(int64_t n_leaves, int cin);
// nbt, gpre, n_groups: the unit-group neighbourhood table, the per-tree
// group prefix and the group count of the preparation (unit voxels' window
// sums are gathered through them).
hipError_t launch_conv_gemm(const ConvArgs& a, const uint64_t* info, const float* wt, float* sbuf,
                            const int32_t* nbt, const int64_t* gpre, const int64_t* n_groups,
                            hipStream_t s);

// Convolution gradients (bias and ReLU excluded): any of dx, dweight, dbias
// may be null.
struct ConvBwdArgs {
  const uint32_t* trees;
  const int64_t* prefix;
  int n, gd, gh, gw;
  int64_t n_trees, n_leaves;
  const float* in;      // forward input [n_leaves][cin] (for dweight)
  int cin;
  const float* weight;  // [cout][cin][27] (for dx)
  int cout;
  const float* dy;      // [n_leaves][cout]
  float* dx;            // [n_leaves][cin]
  float* dweight;       // [cout][cin][27]
  float* dbias;         // [cout]
};
size_t conv_backward_workspace(int64_t n_trees, int64_t n_leaves, int cin, int cout);
bool conv_backward_supported(int cin, int cout);
hipError_t launch_conv_backward(const ConvBwdArgs& a, void* ws, hipStream_t s);

}  // namespace oci
