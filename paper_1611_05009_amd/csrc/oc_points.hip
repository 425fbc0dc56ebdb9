// Grid-octrees from point clouds (the facade segmentation input, Sec. 5):
// points are voxelised into an occupancy grid, the structure is built from
// it as for any occupancy, and every leaf then takes the mean of the
// features of the points inside it (with a binary occupancy channel) and the
// majority of their labels.
#include <hip/hip_runtime.h>

#include "oc_device.h"
#include "oc_internal.h"

using namespace ocd;

namespace {

// Voxel of a point (floor of its coordinates), or false outside the grid.
__device__ __forceinline__ bool point_voxel(const float* __restrict__ pts, const int32_t* __restrict__ batch,
                                            int64_t p, int n, int D, int H, int W, int64_t& b, int& vd,
                                            int& vh, int& vw) {
  const float x = pts[3 * p], y = pts[3 * p + 1], z = pts[3 * p + 2];
  b = batch ? batch[p] : 0;
  // NaN fails every comparison, so it lands outside as well.
  if (!(x >= 0.f && y >= 0.f && z >= 0.f && x < (float)D && y < (float)H && z < (float)W)) return false;
  if (b < 0 || b >= n) return false;
  vd = min((int)x, D - 1);
  vh = min((int)y, H - 1);
  vw = min((int)z, W - 1);
  return true;
}

__global__ void k_zero_bytes(uint8_t* __restrict__ x, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) x[i] = 0;
}

__global__ void k_zero_words(uint32_t* __restrict__ x, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) x[i] = 0u;
}

// occ[b][vd][vh][vw] = 1 for every point inside the grid (same value from
// every writer of a voxel).
__global__ void k_voxelize(const float* __restrict__ pts, const int32_t* __restrict__ batch,
                           int64_t n_pts, int n, int D, int H, int W, uint8_t* __restrict__ occ) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n_pts; p += stride) {
    int64_t b;
    int vd, vh, vw;
    if (point_voxel(pts, batch, p, n, D, H, W, b, vd, vh, vw))
      occ[((b * D + vd) * H + vh) * W + vw] = 1;
  }
}

// Row of the leaf holding each point (Eq. 3 on the leaf's bit index), -1
// outside the grid.
__global__ void k_point_rows(const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix,
                             const float* __restrict__ pts, const int32_t* __restrict__ batch,
                             int64_t n_pts, int n, int gd, int gh, int gw, int32_t* __restrict__ rows) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n_pts; p += stride) {
    int64_t b;
    int vd, vh, vw;
    int32_t r = -1;
    if (point_voxel(pts, batch, p, n, 8 * gd, 8 * gh, 8 * gw, b, vd, vh, vw)) {
      const int64_t t = ((b * gd + (vd >> 3)) * gh + (vh >> 3)) * gw + (vw >> 3);
      const Bits bits = load_bits(trees, t);
      r = (int32_t)(prefix[t] + data_idx(bits, leaf_at(bits, vd & 7, vh & 7, vw & 7)));
    }
    rows[p] = r;
  }
}

// Sums of the point features into out[row][1 + k] and counts per row.
__global__ void k_point_sums(const int32_t* __restrict__ rows, int64_t n_pts,
                             const float* __restrict__ feat, int c, float* __restrict__ out,
                             uint32_t* __restrict__ count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_pts * (c + 1); i += stride) {
    const int64_t p = i / (c + 1);
    const int k = (int)(i - p * (c + 1));
    const int32_t r = rows[p];
    if (r < 0) continue;
    if (k == c) atomicAdd(&count[r], 1u);
    else atomicAdd(&out[(int64_t)r * (c + 1) + 1 + k], feat[p * c + k]);
  }
}

// out[row][0] = 1 if a point fell in the leaf, else 0; out[row][1..c] =
// sums / count (0 without points).
__global__ void k_point_means(const uint32_t* __restrict__ count, int64_t n_leaves, int c,
                              float* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_leaves * (c + 1); i += stride) {
    const int64_t r = i / (c + 1);
    const int k = (int)(i - r * (c + 1));
    const uint32_t m = count[r];
    if (k == 0) out[i] = m > 0 ? 1.f : 0.f;
    else out[i] = m > 0 ? out[i] / (float)m : 0.f;
  }
}

// Label histogram per leaf (hist[row][label]); labels outside [0, L) are
// ignored.
__global__ void k_label_hist(const int32_t* __restrict__ rows, int64_t n_pts,
                             const int32_t* __restrict__ labels, int L, uint32_t* __restrict__ hist) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n_pts; p += stride) {
    const int32_t r = rows[p], l = labels[p];
    if (r >= 0 && l >= 0 && l < L) atomicAdd(&hist[(int64_t)r * L + l], 1u);
  }
}

// The most frequent label of each leaf (the smallest among ties), -1 for a
// leaf without labelled points.
__global__ void k_label_vote(const uint32_t* __restrict__ hist, int64_t n_leaves, int L,
                             int32_t* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n_leaves; r += stride) {
    uint32_t best = 0;
    int32_t arg = -1;
    for (int l = 0; l < L; ++l) {
      const uint32_t h = hist[r * L + l];
      if (h > best) {
        best = h;
        arg = l;
      }
    }
    out[r] = arg;
  }
}

unsigned grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b > 16384) b = 16384;
  if (b < 1) b = 1;
  return (unsigned)b;
}

}  // namespace

namespace oci {

hipError_t launch_voxelize(const float* pts, const int32_t* batch, int64_t n_pts, int n, int gd, int gh,
                           int gw, uint8_t* occ, hipStream_t s) {
  const int D = 8 * gd, H = 8 * gh, W = 8 * gw;
  const int64_t nv = (int64_t)n * D * H * W;
  hipLaunchKernelGGL(k_zero_bytes, dim3(grid_for(nv)), dim3(256), 0, s, occ, nv);
  if (n_pts > 0)
    hipLaunchKernelGGL(k_voxelize, dim3(grid_for(n_pts)), dim3(256), 0, s, pts, batch, n_pts, n, D, H, W,
                       occ);
  return hipGetLastError();
}

hipError_t launch_point_rows(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                             const float* pts, const int32_t* batch, int64_t n_pts, int32_t* rows,
                             hipStream_t s) {
  if (n_pts <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_point_rows, dim3(grid_for(n_pts)), dim3(256), 0, s, trees, prefix, pts, batch,
                     n_pts, n, gd, gh, gw, rows);
  return hipGetLastError();
}

hipError_t launch_point_means(const int32_t* rows, int64_t n_pts, const float* feat, int c,
                              int64_t n_leaves, float* out, uint32_t* count, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_words, dim3(grid_for(n_leaves * (c + 1))), dim3(256), 0, s,
                     reinterpret_cast<uint32_t*>(out), n_leaves * (c + 1));
  hipLaunchKernelGGL(k_zero_words, dim3(grid_for(n_leaves)), dim3(256), 0, s, count, n_leaves);
  if (n_pts > 0)
    hipLaunchKernelGGL(k_point_sums, dim3(grid_for(n_pts * (c + 1))), dim3(256), 0, s, rows, n_pts, feat, c,
                       out, count);
  hipLaunchKernelGGL(k_point_means, dim3(grid_for(n_leaves * (c + 1))), dim3(256), 0, s,
                     (const uint32_t*)count, n_leaves, c, out);
  return hipGetLastError();
}

hipError_t launch_label_vote(const int32_t* rows, int64_t n_pts, const int32_t* labels, int L,
                             int64_t n_leaves, int32_t* out, uint32_t* hist, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_words, dim3(grid_for(n_leaves * L)), dim3(256), 0, s, hist, n_leaves * L);
  if (n_pts > 0)
    hipLaunchKernelGGL(k_label_hist, dim3(grid_for(n_pts)), dim3(256), 0, s, rows, n_pts, labels, L, hist);
  hipLaunchKernelGGL(k_label_vote, dim3(grid_for(n_leaves)), dim3(256), 0, s, (const uint32_t*)hist,
                     n_leaves, L, out);
  return hipGetLastError();
}

}  // namespace oci
