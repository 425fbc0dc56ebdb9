// C ABI entry points: host-side argument checks, workspace carving, launches.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <string>

#include "../../include/octnet_hip.h"
#include "oc_internal.h"

namespace {

// Scratch of oc_build_noalloc: the per-tree leaf counts and the scan's chunk
// sums for up to kNoAllocMaxTrees trees, in a file-scope device array (each
// device the library runs on holds its own copy until the process ends).
// In host code `scratch` only names the symbol; its device address comes
// from hipGetSymbolAddress, once per device, and only that address is used.
constexpr int64_t kNoAllocMaxTrees = 1LL << 22;
constexpr size_t kNoAllocBytes = ((4 * (size_t)kNoAllocMaxTrees + 255) & ~(size_t)255) +
                                 ((8 * ((size_t)kNoAllocMaxTrees / 256 + 2) + 255) & ~(size_t)255) + 1024;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

constexpr int kMaxScratchDevices = 64;

struct ScratchSlot {
  std::once_flag once;
  hipError_t err = hipSuccess;
  void* ptr = nullptr;
};

ScratchSlot g_scratch[kMaxScratchDevices];

// The current device's address of `scratch` (looked up on the first call on
// each device, with that device current).
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  ScratchSlot& sl = g_scratch[dev];
  std::call_once(sl.once, [&sl]() {
    void* p = nullptr;
    sl.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    sl.ptr = p;
  });
  if (sl.err != hipSuccess) return sl.err;
  *out = sl.ptr;
  return hipSuccess;
}

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int hip_fail(hipError_t e, const char* where) {
  return fail(OC_EHIP, "%s: %s", where, hipGetErrorString(e));
}

#define OC_CHECK_HIP(expr, where)                 \
  do {                                            \
    hipError_t _e = (expr);                       \
    if (_e != hipSuccess) return hip_fail(_e, where); \
  } while (0)

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

bool dims_ok(int n, int gd, int gh, int gw) { return n > 0 && gd > 0 && gh > 0 && gw > 0; }

// Voxel and tree counts must fit the int64 index arithmetic of the kernels,
// and a launch grid (blocks of 256 threads over voxels) must fit 2^31 blocks.
bool sizes_ok(int n, int gd, int gh, int gw) {
  const double vox = 512.0 * n * gd * gh * gw;
  return vox < 4.0e12;
}

int64_t n_trees_of(int n, int gd, int gh, int gw) { return (int64_t)n * gd * gh * gw; }

// Scan counts (already in ws) into prefix and read the total back.
int finish_prefix(int64_t nt, int64_t* prefix, int64_t* n_leaves, void* ws, hipStream_t s,
                  const char* where) {
  OC_CHECK_HIP(oci::scan_counts(oci::scan_counts_buffer(ws), nt, prefix, ws, s), where);
  int64_t total = 0;
  OC_CHECK_HIP(hipMemcpyAsync(&total, prefix + nt, sizeof(int64_t), hipMemcpyDeviceToHost, s), where);
  OC_CHECK_HIP(hipStreamSynchronize(s), where);
  *n_leaves = total;
  return OC_OK;
}

}  // namespace

extern "C" {

const char* oc_error_string(int code) {
  switch (code) {
    case OC_OK: return "ok";
    case OC_EINVAL: return "invalid argument";
    case OC_ESTRUCT: return "invalid octree structure";
    case OC_EWORKSPACE: return "workspace too small";
    case OC_EHIP: return "HIP runtime error";
    case OC_EOVERFLOW: return "size overflow";
    default: return "unknown error";
  }
}

const char* oc_last_error(void) { return g_last_error.c_str(); }

int oc_version(void) { return 100; }

size_t oc_structure_workspace(int64_t n_trees) {
  if (n_trees < 0) return 0;
  return oci::scan_workspace(n_trees) + 256;
}

int oc_build(const uint8_t* occ, int n, int gd, int gh, int gw, int rule, uint32_t* trees,
             int64_t* prefix, int64_t* n_leaves, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (!occ || !trees || !prefix || !n_leaves || !ws) return fail(OC_EINVAL, "oc_build: null pointer");
  if (!dims_ok(n, gd, gh, gw)) return fail(OC_EINVAL, "oc_build: non-positive dims");
  if (!sizes_ok(n, gd, gh, gw)) return fail(OC_EOVERFLOW, "oc_build: grid too large");
  if (rule != OC_SPLIT_MIXED && rule != OC_SPLIT_ANY) return fail(OC_EINVAL, "oc_build: bad rule %d", rule);
  const int64_t nt = n_trees_of(n, gd, gh, gw);
  if (ws_bytes < oc_structure_workspace(nt)) return fail(OC_EWORKSPACE, "oc_build: workspace too small");
  hipStream_t s = as_stream(stream);
  OC_CHECK_HIP(oci::launch_build(occ, n, gd, gh, gw, rule, trees, oci::scan_counts_buffer(ws), s),
               "oc_build");
  return finish_prefix(nt, prefix, n_leaves, ws, s, "oc_build");
}

int oc_build_noalloc(const uint8_t* occ, int n, int gd, int gh, int gw, int rule, uint32_t* trees,
                     int64_t* prefix, int64_t* n_leaves, void* stream) {
  g_last_error.clear();
  if (!occ || !trees || !prefix || !n_leaves) return fail(OC_EINVAL, "oc_build_noalloc: null pointer");
  if (!dims_ok(n, gd, gh, gw)) return fail(OC_EINVAL, "oc_build_noalloc: non-positive dims");
  if (!sizes_ok(n, gd, gh, gw)) return fail(OC_EOVERFLOW, "oc_build_noalloc: grid too large");
  if (rule != OC_SPLIT_MIXED && rule != OC_SPLIT_ANY)
    return fail(OC_EINVAL, "oc_build_noalloc: bad rule %d", rule);
  const int64_t nt = n_trees_of(n, gd, gh, gw);
  if (nt > kNoAllocMaxTrees || oci::scan_workspace(nt) > kNoAllocBytes)
    return fail(OC_EOVERFLOW, "oc_build_noalloc: %lld trees exceed the static scratch (at most %lld trees)",
                (long long)nt, (long long)kNoAllocMaxTrees);
  void* ws = nullptr;
  OC_CHECK_HIP(scratch_address(&ws), "oc_build_noalloc");
  hipStream_t s = as_stream(stream);
  OC_CHECK_HIP(oci::launch_build(occ, n, gd, gh, gw, rule, trees, oci::scan_counts_buffer(ws), s),
               "oc_build_noalloc");
  return finish_prefix(nt, prefix, n_leaves, ws, s, "oc_build_noalloc");
}

int oc_prefix(const uint32_t* trees, int64_t n_trees, int64_t* prefix, int64_t* n_leaves, void* ws,
              size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (!trees || !prefix || !n_leaves || !ws) return fail(OC_EINVAL, "oc_prefix: null pointer");
  if (n_trees <= 0) return fail(OC_EINVAL, "oc_prefix: n_trees <= 0");
  if (ws_bytes < oc_structure_workspace(n_trees)) return fail(OC_EWORKSPACE, "oc_prefix: workspace too small");
  hipStream_t s = as_stream(stream);
  // Trees made outside the library enter here: count the non-canonical ones
  // (the counter sits in the workspace's last 256 bytes) with the leaves.
  int32_t* counter = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + oc_structure_workspace(n_trees) - 256);
  OC_CHECK_HIP(hipMemsetAsync(counter, 0, sizeof(int32_t), s), "oc_prefix");
  OC_CHECK_HIP(oci::launch_validate(trees, n_trees, counter, s), "oc_prefix");
  OC_CHECK_HIP(oci::launch_count(trees, n_trees, oci::scan_counts_buffer(ws), s), "oc_prefix");
  int rc = finish_prefix(n_trees, prefix, n_leaves, ws, s, "oc_prefix");
  if (rc != OC_OK) return rc;
  int32_t bad = 0;
  OC_CHECK_HIP(hipMemcpyAsync(&bad, counter, sizeof(int32_t), hipMemcpyDeviceToHost, s), "oc_prefix");
  OC_CHECK_HIP(hipStreamSynchronize(s), "oc_prefix");
  if (bad) return fail(OC_ESTRUCT, "oc_prefix: %d non-canonical trees", bad);
  return OC_OK;
}

int oc_validate(const uint32_t* trees, int64_t n_trees, int64_t* n_bad, void* ws, size_t ws_bytes,
                void* stream) {
  g_last_error.clear();
  if (!trees || !n_bad || !ws) return fail(OC_EINVAL, "oc_validate: null pointer");
  if (n_trees <= 0) return fail(OC_EINVAL, "oc_validate: n_trees <= 0");
  if (ws_bytes < oc_structure_workspace(n_trees)) return fail(OC_EWORKSPACE, "oc_validate: workspace too small");
  hipStream_t s = as_stream(stream);
  int32_t* counter = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + oc_structure_workspace(n_trees) - 256);
  OC_CHECK_HIP(hipMemsetAsync(counter, 0, sizeof(int32_t), s), "oc_validate");
  OC_CHECK_HIP(oci::launch_validate(trees, n_trees, counter, s), "oc_validate");
  int32_t total = 0;
  OC_CHECK_HIP(hipMemcpyAsync(&total, counter, sizeof(int32_t), hipMemcpyDeviceToHost, s), "oc_validate");
  OC_CHECK_HIP(hipStreamSynchronize(s), "oc_validate");
  *n_bad = total;
  return OC_OK;
}

int oc_leaf_index(const uint32_t* trees, const int64_t* prefix, int64_t n_trees, uint64_t* leaf_info,
                  void* stream) {
  g_last_error.clear();
  if (!trees || !prefix || !leaf_info) return fail(OC_EINVAL, "oc_leaf_index: null pointer");
  if (n_trees <= 0) return fail(OC_EINVAL, "oc_leaf_index: n_trees <= 0");
  if (n_trees >= (1LL << 54)) return fail(OC_EOVERFLOW, "oc_leaf_index: too many trees");
  OC_CHECK_HIP(oci::launch_leaf_index(trees, prefix, n_trees, leaf_info, as_stream(stream)),
               "oc_leaf_index");
  return OC_OK;
}

int oc_rowmap(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
              int64_t* rowmap, void* stream) {
  g_last_error.clear();
  if (!trees || !prefix || !rowmap) return fail(OC_EINVAL, "oc_rowmap: null pointer");
  if (!dims_ok(n, gd, gh, gw)) return fail(OC_EINVAL, "oc_rowmap: non-positive dims");
  if (!sizes_ok(n, gd, gh, gw)) return fail(OC_EOVERFLOW, "oc_rowmap: grid too large");
  OC_CHECK_HIP(oci::launch_rowmap(trees, prefix, n, gd, gh, gw, rowmap, as_stream(stream)),
               "oc_rowmap");
  return OC_OK;
}

int oc_oc2ten(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
              const float* data, int c, float* dense, void* stream) {
  g_last_error.clear();
  if (!trees || !prefix || !data || !dense) return fail(OC_EINVAL, "oc_oc2ten: null pointer");
  if (!dims_ok(n, gd, gh, gw) || c <= 0) return fail(OC_EINVAL, "oc_oc2ten: non-positive dims");
  if (!sizes_ok(n, gd, gh, gw)) return fail(OC_EOVERFLOW, "oc_oc2ten: grid too large");
  OC_CHECK_HIP(oci::launch_oc2ten(trees, prefix, n, gd, gh, gw, data, c, dense, as_stream(stream)),
               "oc_oc2ten");
  return OC_OK;
}

int oc_ten2oc(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
              const float* dense, int c, int pool, float* data, void* stream) {
  g_last_error.clear();
  if (!trees || !prefix || !data || !dense) return fail(OC_EINVAL, "oc_ten2oc: null pointer");
  if (!dims_ok(n, gd, gh, gw) || c <= 0) return fail(OC_EINVAL, "oc_ten2oc: non-positive dims");
  if (pool != OC_POOL_AVG && pool != OC_POOL_MAX) return fail(OC_EINVAL, "oc_ten2oc: bad pool %d", pool);
  if (!sizes_ok(n, gd, gh, gw)) return fail(OC_EOVERFLOW, "oc_ten2oc: grid too large");
  OC_CHECK_HIP(oci::launch_ten2oc(trees, prefix, n, gd, gh, gw, dense, c, pool, data,
                                  as_stream(stream)),
               "oc_ten2oc");
  return OC_OK;
}

int oc_conv3x3x3_workspace(int64_t n_trees, int64_t n_leaves, int cin, int cout, size_t* bytes) {
  g_last_error.clear();
  if (!bytes) return fail(OC_EINVAL, "oc_conv3x3x3_workspace: null pointer");
  if (n_trees <= 0 || n_leaves <= 0 || cin <= 0 || cout <= 0)
    return fail(OC_EINVAL, "oc_conv3x3x3_workspace: non-positive size");
  *bytes = oci::conv_workspace(n_trees, n_leaves, cin, cout);
  return OC_OK;
}

int oc_conv3x3x3_workspace_exact(const uint32_t* trees, int n, int gd, int gh, int gw, int64_t n_leaves,
                                 int cin, int cout, size_t* bytes, void* scratch, void* stream) {
  g_last_error.clear();
  if (!trees || !bytes || !scratch) return fail(OC_EINVAL, "oc_conv3x3x3_workspace_exact: null pointer");
  if (!dims_ok(n, gd, gh, gw) || n_leaves <= 0 || cin <= 0 || cout <= 0)
    return fail(OC_EINVAL, "oc_conv3x3x3_workspace_exact: non-positive size");
  const int64_t nt = n_trees_of(n, gd, gh, gw);
  hipStream_t s = as_stream(stream);
  unsigned long long* count = static_cast<unsigned long long*>(scratch);
  OC_CHECK_HIP(oci::launch_count_slots(trees, nt, count, s), "oc_conv3x3x3_workspace_exact");
  unsigned long long slots = 0;
  OC_CHECK_HIP(hipMemcpyAsync(&slots, count, sizeof(slots), hipMemcpyDeviceToHost, s),
               "oc_conv3x3x3_workspace_exact");
  OC_CHECK_HIP(hipStreamSynchronize(s), "oc_conv3x3x3_workspace_exact");
  *bytes = oci::conv_workspace_slots(nt, n_leaves, cin, cout, (int64_t)slots);
  return OC_OK;
}

int oc_conv3x3x3_workspace_slots(int64_t n_trees, int64_t n_leaves, int cin, int cout, int64_t slots,
                                 size_t* bytes) {
  g_last_error.clear();
  if (!bytes) return fail(OC_EINVAL, "oc_conv3x3x3_workspace_slots: null pointer");
  if (n_trees <= 0 || n_leaves <= 0 || cin <= 0 || cout <= 0)
    return fail(OC_EINVAL, "oc_conv3x3x3_workspace_slots: non-positive size");
  *bytes = oci::conv_workspace_slots(n_trees, n_leaves, cin, cout, slots);
  return OC_OK;
}

int oc_conv3x3x3_workspace_capacity(int64_t n_trees, int64_t n_leaves, int cin, int cout, size_t ws_bytes,
                                    int64_t* slots) {
  g_last_error.clear();
  if (!slots) return fail(OC_EINVAL, "oc_conv3x3x3_workspace_capacity: null pointer");
  if (n_trees <= 0 || n_leaves <= 0 || cin <= 0 || cout <= 0)
    return fail(OC_EINVAL, "oc_conv3x3x3_workspace_capacity: non-positive size");
  const int64_t cap = oci::conv_slot_capacity(n_trees, n_leaves, cin, cout, ws_bytes);
  if (cap < 0) return fail(OC_EWORKSPACE, "oc_conv3x3x3_workspace_capacity: below the one-slot size");
  *slots = cap;
  return OC_OK;
}

int oc_conv3x3x3_mfma_supported(int cin, int cout) { return oci::conv_mfma_supported(cin, cout) ? 1 : 0; }

namespace {

// Shared argument checks of the convolution entry points; fills `a`.
int conv_args(const char* who, const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
              int gw, int64_t n_leaves, int cin, int cout, size_t ws_bytes, const void* ws,
              oci::ConvArgs* a) {
  if (!trees || !prefix || !ws) return fail(OC_EINVAL, "%s: null pointer", who);
  if (!dims_ok(n, gd, gh, gw)) return fail(OC_EINVAL, "%s: non-positive dims", who);
  if (cin <= 0 || cout <= 0 || cin > 256 || cout > 4096)
    return fail(OC_EINVAL, "%s: channels (%d, %d) outside [1,256] x [1,4096]", who, cin, cout);
  if (n_leaves <= 0) return fail(OC_EINVAL, "%s: n_leaves <= 0", who);
  if (n_leaves >= (1LL << 31)) return fail(OC_EOVERFLOW, "%s: n_leaves >= 2^31", who);
  const int64_t nt = n_trees_of(n, gd, gh, gw);
  if (n_leaves > 512 * nt) return fail(OC_EINVAL, "%s: n_leaves > 512 * n_trees", who);
  const int64_t cap = oci::conv_slot_capacity(nt, n_leaves, cin, cout, ws_bytes);
  if (cap < 0)
    return fail(OC_EWORKSPACE, "%s: workspace %zu < %zu", who, ws_bytes,
                oci::conv_workspace_slots(nt, n_leaves, cin, cout, 1));
  *a = oci::ConvArgs();
  a->slot_cap = cap;
  a->trees = trees; a->prefix = prefix;
  a->n = n; a->gd = gd; a->gh = gh; a->gw = gw;
  a->n_trees = nt; a->n_leaves = n_leaves;
  a->cin = cin; a->cout = cout;
  return OC_OK;
}

int conv_impl(const char* who, int impl, int64_t n_leaves, int cin, int cout, int* use) {
  if (impl != OC_CONV_AUTO && impl != OC_CONV_GENERIC && impl != OC_CONV_MFMA && impl != OC_CONV_GEMM &&
      impl != OC_CONV_TRUNCATED)
    return fail(OC_EINVAL, "%s: bad impl %d", who, impl);
  const bool mfma_ok = oci::conv_mfma_supported(cin, cout);
  if (impl == OC_CONV_MFMA && !mfma_ok)
    return fail(OC_EINVAL, "%s: no MFMA kernel for (%d, %d)", who, cin, cout);
  *use = impl == OC_CONV_AUTO ? oci::conv_auto_impl(n_leaves, cin, cout) : impl;
  return OC_OK;
}

}  // namespace

int oc_conv3x3x3_prepare(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                         int64_t n_leaves, const float* weight, int cin, int cout, void* ws,
                         size_t ws_bytes, void* stream) {
  g_last_error.clear();
  oci::ConvArgs a;
  int rc = conv_args("oc_conv3x3x3_prepare", trees, prefix, n, gd, gh, gw, n_leaves, cin, cout,
                     ws_bytes, ws, &a);
  if (rc != OC_OK) return rc;
  if (!weight) return fail(OC_EINVAL, "oc_conv3x3x3_prepare: null weight");
  a.weight = weight;
  OC_CHECK_HIP(oci::launch_conv_prepare(a, ws, as_stream(stream)), "oc_conv3x3x3_prepare");
  return OC_OK;
}

int oc_conv3x3x3_execute(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                         int64_t n_leaves, const float* in, int cin, const float* bias, int cout,
                         int relu, float* out, void* ws, size_t ws_bytes, int impl,
                         void* stream) {
  g_last_error.clear();
  oci::ConvArgs a;
  int rc = conv_args("oc_conv3x3x3_execute", trees, prefix, n, gd, gh, gw, n_leaves, cin, cout,
                     ws_bytes, ws, &a);
  if (rc != OC_OK) return rc;
  if (!in || !out) return fail(OC_EINVAL, "oc_conv3x3x3_execute: null pointer");
  int use = 0;
  rc = conv_impl("oc_conv3x3x3_execute", impl, n_leaves, cin, cout, &use);
  if (rc != OC_OK) return rc;
  if (use == OC_CONV_TRUNCATED)
    return fail(OC_EINVAL, "oc_conv3x3x3_execute: OC_CONV_TRUNCATED runs through oc_conv3x3x3_ex");
  a.in = in; a.bias = bias; a.relu = relu ? 1 : 0; a.out = out;
  OC_CHECK_HIP(oci::launch_conv_execute(a, ws, use, as_stream(stream)), "oc_conv3x3x3_execute");
  return OC_OK;
}

int oc_conv3x3x3_ex(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                    int64_t n_leaves, const float* in, int cin, const float* weight,
                    const float* bias, int cout, int relu, float* out, void* ws, size_t ws_bytes,
                    int impl, void* stream) {
  g_last_error.clear();
  oci::ConvArgs a;
  int rc = conv_args("oc_conv3x3x3", trees, prefix, n, gd, gh, gw, n_leaves, cin, cout, ws_bytes, ws,
                     &a);
  if (rc != OC_OK) return rc;
  if (!in || !weight || !out) return fail(OC_EINVAL, "oc_conv3x3x3: null pointer");
  int use = 0;
  rc = conv_impl("oc_conv3x3x3", impl, n_leaves, cin, cout, &use);
  if (rc != OC_OK) return rc;
  a.in = in; a.weight = weight; a.bias = bias; a.relu = relu ? 1 : 0; a.out = out;
  hipStream_t s = as_stream(stream);
  if (use == OC_CONV_TRUNCATED) {
    // Needs only the leaf index, at the start of the workspace.
    OC_CHECK_HIP(oci::launch_conv_truncated(a, static_cast<uint64_t*>(ws), s), "oc_conv3x3x3");
    return OC_OK;
  }
  OC_CHECK_HIP(oci::launch_conv_prepare(a, ws, s), "oc_conv3x3x3");
  OC_CHECK_HIP(oci::launch_conv_execute(a, ws, use, s), "oc_conv3x3x3");
  return OC_OK;
}

int oc_conv3x3x3(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                 int64_t n_leaves, const float* in, int cin, const float* weight, const float* bias,
                 int cout, int relu, float* out, void* ws, size_t ws_bytes, void* stream) {
  return oc_conv3x3x3_ex(trees, prefix, n, gd, gh, gw, n_leaves, in, cin, weight, bias, cout, relu,
                         out, ws, ws_bytes, OC_CONV_AUTO, stream);
}

int oc_pool2_structure(const uint32_t* in_trees, int n, int gd, int gh, int gw, uint32_t* out_trees,
                       int64_t* out_prefix, int64_t* out_n_leaves, void* ws, size_t ws_bytes,
                       void* stream) {
  g_last_error.clear();
  if (!in_trees || !out_trees || !out_prefix || !out_n_leaves || !ws)
    return fail(OC_EINVAL, "oc_pool2_structure: null pointer");
  if (!dims_ok(n, gd, gh, gw)) return fail(OC_EINVAL, "oc_pool2_structure: non-positive dims");
  if ((gd | gh | gw) & 1) return fail(OC_EINVAL, "oc_pool2_structure: odd tree grid %dx%dx%d", gd, gh, gw);
  const int64_t no = (int64_t)n * (gd / 2) * (gh / 2) * (gw / 2);
  if (ws_bytes < oc_structure_workspace(no)) return fail(OC_EWORKSPACE, "oc_pool2_structure: workspace too small");
  hipStream_t s = as_stream(stream);
  OC_CHECK_HIP(oci::launch_pool_structure(in_trees, n, gd, gh, gw, out_trees,
                                          oci::scan_counts_buffer(ws), s),
               "oc_pool2_structure");
  return finish_prefix(no, out_prefix, out_n_leaves, ws, s, "oc_pool2_structure");
}

int oc_pool2_max(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh, int gw,
                 const float* in, int c, const uint32_t* out_trees, const int64_t* out_prefix,
                 float* out, void* stream) {
  g_last_error.clear();
  if (!in_trees || !in_prefix || !in || !out_trees || !out_prefix || !out)
    return fail(OC_EINVAL, "oc_pool2_max: null pointer");
  if (!dims_ok(n, gd, gh, gw) || c <= 0) return fail(OC_EINVAL, "oc_pool2_max: non-positive dims");
  if ((gd | gh | gw) & 1) return fail(OC_EINVAL, "oc_pool2_max: odd tree grid");
  OC_CHECK_HIP(oci::launch_pool_max(in_trees, in_prefix, n, gd, gh, gw, in, c, out_trees, out_prefix,
                                    out, as_stream(stream)),
               "oc_pool2_max");
  return OC_OK;
}

int oc_unpool2_structure(const uint32_t* in_trees, int n, int gd, int gh, int gw,
                         const uint32_t* guide_trees, uint32_t* out_trees, int64_t* out_prefix,
                         int64_t* out_n_leaves, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (!in_trees || !out_trees || !out_prefix || !out_n_leaves || !ws)
    return fail(OC_EINVAL, "oc_unpool2_structure: null pointer");
  if (!dims_ok(n, gd, gh, gw)) return fail(OC_EINVAL, "oc_unpool2_structure: non-positive dims");
  if (!sizes_ok(n, 2 * gd, 2 * gh, 2 * gw)) return fail(OC_EOVERFLOW, "oc_unpool2_structure: grid too large");
  const int64_t no = 8LL * n * gd * gh * gw;
  if (ws_bytes < oc_structure_workspace(no)) return fail(OC_EWORKSPACE, "oc_unpool2_structure: workspace too small");
  hipStream_t s = as_stream(stream);
  // The mismatch flag of the guided check sits in the last 256 bytes.
  int32_t* mismatch = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + oc_structure_workspace(no) - 256);
  if (guide_trees) OC_CHECK_HIP(hipMemsetAsync(mismatch, 0, sizeof(int32_t), s), "oc_unpool2_structure");
  OC_CHECK_HIP(oci::launch_unpool_structure(in_trees, guide_trees, n, gd, gh, gw, out_trees,
                                            oci::scan_counts_buffer(ws), mismatch, s),
               "oc_unpool2_structure");
  int rc = finish_prefix(no, out_prefix, out_n_leaves, ws, s, "oc_unpool2_structure");
  if (rc != OC_OK) return rc;
  if (guide_trees) {
    int32_t bad = 0;
    OC_CHECK_HIP(hipMemcpyAsync(&bad, mismatch, sizeof(int32_t), hipMemcpyDeviceToHost, s),
                 "oc_unpool2_structure");
    OC_CHECK_HIP(hipStreamSynchronize(s), "oc_unpool2_structure");
    if (bad) return fail(OC_ESTRUCT, "oc_unpool2_structure: guide does not pool to the input (%d trees)", bad);
  }
  return OC_OK;
}

int oc_unpool2(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh, int gw,
               const float* in, int c, const uint32_t* out_trees, const int64_t* out_prefix,
               float* out, void* stream) {
  g_last_error.clear();
  if (!in_trees || !in_prefix || !in || !out_trees || !out_prefix || !out)
    return fail(OC_EINVAL, "oc_unpool2: null pointer");
  if (!dims_ok(n, gd, gh, gw) || c <= 0) return fail(OC_EINVAL, "oc_unpool2: non-positive dims");
  OC_CHECK_HIP(oci::launch_unpool(in_trees, in_prefix, n, gd, gh, gw, in, c, out_trees, out_prefix,
                                  out, as_stream(stream)),
               "oc_unpool2");
  return OC_OK;
}

int oc_relu(float* data, int64_t count, void* stream) {
  g_last_error.clear();
  if (!data) return fail(OC_EINVAL, "oc_relu: null pointer");
  if (count < 0) return fail(OC_EINVAL, "oc_relu: negative count");
  OC_CHECK_HIP(oci::launch_relu(data, count, as_stream(stream)), "oc_relu");
  return OC_OK;
}

int oc_conv3x3x3_backward_workspace(int64_t n_trees, int64_t n_leaves, int cin, int cout,
                                    size_t* bytes) {
  g_last_error.clear();
  if (!bytes) return fail(OC_EINVAL, "oc_conv3x3x3_backward_workspace: null pointer");
  if (n_trees <= 0 || n_leaves <= 0 || cin <= 0 || cout <= 0)
    return fail(OC_EINVAL, "oc_conv3x3x3_backward_workspace: non-positive size");
  *bytes = oci::conv_backward_workspace(n_trees, n_leaves, cin, cout);
  return OC_OK;
}

int oc_conv3x3x3_backward(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
                          int gw, int64_t n_leaves, const float* in, int cin, const float* weight,
                          int cout, const float* dout, float* din, float* dweight, float* dbias,
                          void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  const char* who = "oc_conv3x3x3_backward";
  if (!trees || !prefix || !ws || !dout) return fail(OC_EINVAL, "%s: null pointer", who);
  if (din && !weight) return fail(OC_EINVAL, "%s: din needs weight", who);
  if (dweight && !in) return fail(OC_EINVAL, "%s: dweight needs in", who);
  if (!dims_ok(n, gd, gh, gw)) return fail(OC_EINVAL, "%s: non-positive dims", who);
  if (cin <= 0 || cout <= 0 || cin > 256 || cout > 256)
    return fail(OC_EINVAL, "%s: channels (%d, %d) outside [1,256] x [1,256]", who, cin, cout);
  if (n_leaves <= 0) return fail(OC_EINVAL, "%s: n_leaves <= 0", who);
  if (n_leaves >= (1LL << 31)) return fail(OC_EOVERFLOW, "%s: n_leaves >= 2^31", who);
  const int64_t nt = n_trees_of(n, gd, gh, gw);
  if (n_leaves > 512 * nt) return fail(OC_EINVAL, "%s: n_leaves > 512 * n_trees", who);
  const size_t need = oci::conv_backward_workspace(nt, n_leaves, cin, cout);
  if (ws_bytes < need) return fail(OC_EWORKSPACE, "%s: workspace %zu < %zu", who, ws_bytes, need);
  if (dweight && !oci::conv_backward_supported(cin, cout))
    return fail(OC_EINVAL, "%s: no weight-gradient kernel for (%d, %d)", who, cin, cout);
  oci::ConvBwdArgs a;
  a.trees = trees; a.prefix = prefix;
  a.n = n; a.gd = gd; a.gh = gh; a.gw = gw;
  a.n_trees = nt; a.n_leaves = n_leaves;
  a.in = in; a.cin = cin; a.weight = weight; a.cout = cout;
  a.dy = dout; a.dx = din; a.dweight = dweight; a.dbias = dbias;
  OC_CHECK_HIP(oci::launch_conv_backward(a, ws, as_stream(stream)), who);
  return OC_OK;
}

int oc_pool2_max_backward(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh,
                          int gw, const float* in, int c, const uint32_t* out_trees,
                          const int64_t* out_prefix, const float* dout, float* din, void* stream) {
  g_last_error.clear();
  if (!in_trees || !in_prefix || !in || !out_trees || !out_prefix || !dout || !din)
    return fail(OC_EINVAL, "oc_pool2_max_backward: null pointer");
  if (!dims_ok(n, gd, gh, gw) || c <= 0)
    return fail(OC_EINVAL, "oc_pool2_max_backward: non-positive dims");
  if ((gd | gh | gw) & 1) return fail(OC_EINVAL, "oc_pool2_max_backward: odd tree grid");
  OC_CHECK_HIP(oci::launch_pool_max_bwd(in_trees, in_prefix, n, gd, gh, gw, in, c, out_trees,
                                        out_prefix, dout, din, as_stream(stream)),
               "oc_pool2_max_backward");
  return OC_OK;
}

int oc_unpool2_backward(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh,
                        int gw, int64_t in_n_leaves, int c, const uint32_t* out_trees,
                        const int64_t* out_prefix, const float* dout, float* din, void* stream) {
  g_last_error.clear();
  if (!in_trees || !in_prefix || !out_trees || !out_prefix || !dout || !din)
    return fail(OC_EINVAL, "oc_unpool2_backward: null pointer");
  if (!dims_ok(n, gd, gh, gw) || c <= 0 || in_n_leaves <= 0)
    return fail(OC_EINVAL, "oc_unpool2_backward: non-positive dims");
  if (in_n_leaves > 512 * n_trees_of(n, gd, gh, gw))
    return fail(OC_EINVAL, "oc_unpool2_backward: in_n_leaves > 512 * n_trees");
  if (!sizes_ok(n, 2 * gd, 2 * gh, 2 * gw)) return fail(OC_EOVERFLOW, "oc_unpool2_backward: grid too large");
  OC_CHECK_HIP(oci::launch_unpool_bwd(in_trees, in_prefix, n, gd, gh, gw, in_n_leaves, c, out_trees,
                                      out_prefix, dout, din, as_stream(stream)),
               "oc_unpool2_backward");
  return OC_OK;
}

int oc_relu_backward(const float* out, const float* dout, float* din, int64_t count, void* stream) {
  g_last_error.clear();
  if (count < 0) return fail(OC_EINVAL, "oc_relu_backward: negative count");
  if (count == 0) return OC_OK;
  if (!out || !dout || !din) return fail(OC_EINVAL, "oc_relu_backward: null pointer");
  OC_CHECK_HIP(oci::launch_relu_bwd(out, dout, din, count, as_stream(stream)), "oc_relu_backward");
  return OC_OK;
}

int oc_concat(const float* a, int ca, const float* b, int cb, int64_t n_rows, float* out, void* stream) {
  g_last_error.clear();
  if (ca <= 0 || cb <= 0 || n_rows < 0) return fail(OC_EINVAL, "oc_concat: non-positive size");
  if (n_rows == 0) return OC_OK;
  if (!a || !b || !out) return fail(OC_EINVAL, "oc_concat: null pointer");
  if ((double)n_rows * (ca + cb) >= 9.0e18) return fail(OC_EOVERFLOW, "oc_concat: too large");
  OC_CHECK_HIP(oci::launch_concat(a, ca, b, cb, n_rows, out, as_stream(stream)), "oc_concat");
  return OC_OK;
}

int oc_concat_backward(const float* dout, int ca, int cb, int64_t n_rows, float* da, float* db,
                       void* stream) {
  g_last_error.clear();
  if (ca <= 0 || cb <= 0 || n_rows < 0) return fail(OC_EINVAL, "oc_concat_backward: non-positive size");
  if (n_rows == 0 || (!da && !db)) return OC_OK;
  if (!dout) return fail(OC_EINVAL, "oc_concat_backward: null pointer");
  OC_CHECK_HIP(oci::launch_split(dout, ca, cb, n_rows, da, db, as_stream(stream)), "oc_concat_backward");
  return OC_OK;
}

int oc_add(const float* a, const float* b, float* out, int64_t count, void* stream) {
  g_last_error.clear();
  if (count < 0) return fail(OC_EINVAL, "oc_add: negative count");
  if (count == 0) return OC_OK;
  if (!a || !b || !out) return fail(OC_EINVAL, "oc_add: null pointer");
  OC_CHECK_HIP(oci::launch_add(a, b, out, count, as_stream(stream)), "oc_add");
  return OC_OK;
}

int oc_points_voxelize(const float* pts, const int32_t* batch, int64_t n_pts, int n, int gd, int gh,
                       int gw, uint8_t* occ, void* stream) {
  g_last_error.clear();
  if (!occ || (n_pts > 0 && !pts)) return fail(OC_EINVAL, "oc_points_voxelize: null pointer");
  if (!dims_ok(n, gd, gh, gw) || n_pts < 0) return fail(OC_EINVAL, "oc_points_voxelize: non-positive dims");
  if (!sizes_ok(n, gd, gh, gw)) return fail(OC_EOVERFLOW, "oc_points_voxelize: grid too large");
  OC_CHECK_HIP(oci::launch_voxelize(pts, batch, n_pts, n, gd, gh, gw, occ, as_stream(stream)),
               "oc_points_voxelize");
  return OC_OK;
}

int oc_points_leaf_rows(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                        const float* pts, const int32_t* batch, int64_t n_pts, int32_t* rows,
                        void* stream) {
  g_last_error.clear();
  if (n_pts < 0 || !dims_ok(n, gd, gh, gw)) return fail(OC_EINVAL, "oc_points_leaf_rows: bad size");
  if (n_pts == 0) return OC_OK;
  if (!trees || !prefix || !pts || !rows) return fail(OC_EINVAL, "oc_points_leaf_rows: null pointer");
  if (!sizes_ok(n, gd, gh, gw)) return fail(OC_EOVERFLOW, "oc_points_leaf_rows: grid too large");
  OC_CHECK_HIP(oci::launch_point_rows(trees, prefix, n, gd, gh, gw, pts, batch, n_pts, rows,
                                      as_stream(stream)),
               "oc_points_leaf_rows");
  return OC_OK;
}

size_t oc_points_workspace(int64_t n_leaves, int n_labels) {
  const int64_t per = n_labels > 1 ? n_labels : 1;
  return (size_t)(n_leaves > 0 ? n_leaves : 0) * (size_t)per * sizeof(uint32_t) + 256;
}

int oc_points_average(const int32_t* rows, int64_t n_pts, const float* feat, int c, int64_t n_leaves,
                      float* out, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (n_pts < 0 || c < 0 || n_leaves <= 0) return fail(OC_EINVAL, "oc_points_average: bad size");
  if (!out || !ws || (n_pts > 0 && (!rows || (c > 0 && !feat))))
    return fail(OC_EINVAL, "oc_points_average: null pointer");
  if (ws_bytes < oc_points_workspace(n_leaves, 1))
    return fail(OC_EWORKSPACE, "oc_points_average: workspace too small");
  OC_CHECK_HIP(oci::launch_point_means(rows, n_pts, feat, c, n_leaves, out, static_cast<uint32_t*>(ws),
                                       as_stream(stream)),
               "oc_points_average");
  return OC_OK;
}

int oc_points_vote(const int32_t* rows, int64_t n_pts, const int32_t* labels, int n_labels,
                   int64_t n_leaves, int32_t* out, void* ws, size_t ws_bytes, void* stream) {
  g_last_error.clear();
  if (n_pts < 0 || n_labels <= 0 || n_leaves <= 0) return fail(OC_EINVAL, "oc_points_vote: bad size");
  if (!out || !ws || (n_pts > 0 && (!rows || !labels))) return fail(OC_EINVAL, "oc_points_vote: null pointer");
  if (ws_bytes < oc_points_workspace(n_leaves, n_labels))
    return fail(OC_EWORKSPACE, "oc_points_vote: workspace too small");
  OC_CHECK_HIP(oci::launch_label_vote(rows, n_pts, labels, n_labels, n_leaves, out,
                                      static_cast<uint32_t*>(ws), as_stream(stream)),
               "oc_points_vote");
  return OC_OK;
}

}  // extern "C"
