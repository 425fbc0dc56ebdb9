// The paper's efficient convolution for large cells (supplement, "Efficient
// Convolution"), as an alternative kernel: inside a leaf the input is
// constant, so the kernel is applied once to the leaf's own value and scaled
// by the cell volume, and only the taps of boundary voxels that reach
// outside the cell (19 at a corner, 15 along an edge, 9 on a face) are
// evaluated with the neighbouring values, as corrections x(u + delta) - x_l.
// For an 8^3 cell that is 27 + 8*19 + 12*6*15 + 6*6^2*9 = 3203 products per
// channel pair instead of 27 * 8^3.  The result is Eq. 8 (average pooling)
// up to rounding.  VALU only: it is kept as the paper's scheme, next to the
// window-sum kernels that need 27 products per pair for any cell size.
#include <hip/hip_runtime.h>

#include "oc_device.h"
#include "oc_internal.h"

using namespace ocd;

namespace {

// Row of the leaf holding global voxel (vd, vh, vw) of sample n, -1 outside.
__device__ __forceinline__ int64_t voxel_row(const uint32_t* __restrict__ trees,
                                             const int64_t* __restrict__ prefix, int64_t n, int gd,
                                             int gh, int gw, int vd, int vh, int vw) {
  if (vd < 0 || vh < 0 || vw < 0 || vd >= 8 * gd || vh >= 8 * gh || vw >= 8 * gw) return -1;
  const int64_t t = ((n * gd + (vd >> 3)) * gh + (vh >> 3)) * gw + (vw >> 3);
  const Bits b = load_bits(trees, t);
  return prefix[t] + data_idx(b, leaf_at(b, vd & 7, vh & 7, vw & 7));
}

// One wave per leaf, lanes over output channels (co0 + lane).  LDS per wave:
// the leaf's own row and the current neighbour row, cin floats each.
__global__ void __launch_bounds__(256) k_conv_truncated(
    const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix,
    const uint64_t* __restrict__ info, int64_t n_leaves, int gd, int gh, int gw,
    const float* __restrict__ in, int cin, const float* __restrict__ w,
    const float* __restrict__ bias, int cout, int relu, float* __restrict__ out) {
  extern __shared__ float lds[];
  const int wv = threadIdx.x >> 6, lane = lane_id();
  float* xl = lds + (size_t)wv * 2 * cin;
  float* xn = xl + cin;
  for (int64_t row = (int64_t)blockIdx.x * 4 + wv; row < n_leaves; row += (int64_t)gridDim.x * 4) {
    const uint64_t inf = info[row];
    const TreePos p = tree_pos((int64_t)(inf >> 10), gd, gh, gw);
    const Cell c = cell_of((int)(inf & 1023u));
    const int s = c.size;
    const int od = 8 * p.d + c.d, oh = 8 * p.h + c.h, ow = 8 * p.w + c.w;
    for (int ci = lane; ci < cin; ci += 64) xl[ci] = in[row * cin + ci];
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    for (int co0 = 0; co0 < cout; co0 += 64) {
      const int co = co0 + lane;
      const bool live = co < cout;
      const float* wc = w + (int64_t)(live ? co : 0) * cin * 27;
      // The constant part: the full kernel applied to x_l (times |l|, which
      // the average divides out again, so it is kept apart).
      float cst = 0.f;
      for (int ci = 0; ci < cin; ++ci) {
        float ws = 0.f;
        for (int t = 0; t < 27; ++t) ws += wc[ci * 27 + t];
        cst = fmaf(ws, xl[ci], cst);
      }
      float acc = 0.f;
      // Corrections at boundary voxels u (some coordinate at 0 or s - 1),
      // for every tap that leaves the cell.
      for (int ud = 0; ud < s; ++ud)
        for (int uh = 0; uh < s; ++uh)
          for (int uw = 0; uw < s; ++uw) {
            const bool bnd = ud == 0 || uh == 0 || uw == 0 || ud == s - 1 || uh == s - 1 || uw == s - 1;
            if (!bnd) {
              uw = s - 2;  // skip to the far face of this row
              continue;
            }
            for (int t = 0; t < 27; ++t) {
              const int dd = t / 9 - 1, dh = (t / 3) % 3 - 1, dw = t % 3 - 1;
              const int qd = ud + dd, qh = uh + dh, qw = uw + dw;
              if (qd >= 0 && qh >= 0 && qw >= 0 && qd < s && qh < s && qw < s) continue;
              const int64_t nr = voxel_row(trees, prefix, p.n, gd, gh, gw, od + qd, oh + qh, ow + qw);
              __builtin_amdgcn_wave_barrier();
              for (int ci = lane; ci < cin; ci += 64) xn[ci] = nr >= 0 ? in[nr * cin + ci] : 0.f;
              __builtin_amdgcn_wave_barrier();
              __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
              // Eq. 7: tap 1 - delta multiplies x(u + delta).
              const int tap = (1 - dd) * 9 + (1 - dh) * 3 + (1 - dw);
              for (int ci = 0; ci < cin; ++ci) acc = fmaf(wc[ci * 27 + tap], xn[ci] - xl[ci], acc);
            }
          }
      if (live) {
        float v = cst + acc / (float)(s * s * s) + (bias ? bias[co] : 0.f);
        if (relu) v = fmaxf(v, 0.f);
        out[row * cout + co] = v;
      }
    }
    __builtin_amdgcn_wave_barrier();  // xl is rewritten for the next leaf
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  }
}

}  // namespace

namespace oci {

hipError_t launch_conv_truncated(const ConvArgs& a, uint64_t* info, hipStream_t s) {
  hipError_t e = launch_leaf_index(a.trees, a.prefix, a.n_trees, info, s);
  if (e != hipSuccess) return e;
  int64_t blocks = (a.n_leaves + 3) / 4;
  if (blocks > 65536) blocks = 65536;
  const size_t smem = sizeof(float) * 4 * 2 * (size_t)a.cin;
  hipLaunchKernelGGL(k_conv_truncated, dim3((unsigned)blocks), dim3(256), smem, s, a.trees, a.prefix,
                     (const uint64_t*)info, a.n_leaves, a.gd, a.gh, a.gw, a.in, a.cin, a.weight, a.bias,
                     a.cout, a.relu, a.out);
  return hipGetLastError();
}

}  // namespace oci
