// Feature kernels: oc2ten / ten2oc (Eq. 4-5), 2x2x2 max-pooling data
// (Eq. 10), 2x2x2 unpooling data (Eq. 12 and its guided variant), ReLU.
#include "oc_internal.h"

using namespace ocd;

namespace {

template <int V> struct VecF;
template <> struct VecF<1> { typedef float type; };
template <> struct VecF<4> { typedef float4 type; };

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// Eq. 4: one thread per voxel copies the c features of the leaf holding it.
__global__ void k_oc2ten(const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix,
                         int64_t n_vox, int gd, int gh, int gw, const float* __restrict__ data,
                         int c, float* __restrict__ dense) {
  const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= n_vox) return;
  const int64_t W = 8LL * gw, H = 8LL * gh, D = 8LL * gd;
  int64_t r = v;
  const int vw = (int)(r % W); r /= W;
  const int vh = (int)(r % H); r /= H;
  const int vd = (int)(r % D); r /= D;
  const int64_t t = ((r * gd + (vd >> 3)) * gh + (vh >> 3)) * gw + (vw >> 3);
  const Bits b = load_bits(trees, t);
  const int64_t row = prefix[t] + data_idx(b, leaf_at(b, vd & 7, vh & 7, vw & 7));
  const float* src = data + row * c;
  float* dst = dense + v * c;
  for (int k = 0; k < c; ++k) dst[k] = src[k];
}

// Eq. 5: one wave per tree.  Lane l = 8 h + w takes the voxel column (h, w)
// of the tree and reads its 8 voxels along d, c channels each: 8 lanes read
// 8 consecutive voxels of a grid row, so a load instruction covers 8 rows
// (16-byte loads where c % 4 == 0).  The cell values at every level come
// from that one read: the 2^3 blocks by adding d pairs in the lane, then
// lanes w ^ 1 and h ^ 1; the 4^3 blocks from pairs of those, lanes w ^ 2
// and h ^ 2; the tree from lanes w ^ 4 and h ^ 4 -- sums in double for the
// average, maxima for max pooling, in a fixed order.  The leaf holding each
// voxel comes from the split bits; the lane holding the leaf's first voxel
// writes its row (Eq. 3 gives the row).
template <bool VEC4>
__global__ void __launch_bounds__(256) k_ten2oc(const uint32_t* __restrict__ trees,
                                                const int64_t* __restrict__ prefix, int64_t n_trees,
                                                int gd, int gh, int gw,
                                                const float* __restrict__ dense, int c, int pool,
                                                float* __restrict__ data) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_trees) return;  // whole wave exits together
  const Bits b = load_bits(trees, t);
  const TreePos p = tree_pos(t, gd, gh, gw);
  const int64_t W = 8LL * gw, H = 8LL * gh, D = 8LL * gd;
  const int64_t row0 = prefix[t];
  const int lane = lane_id(), lh = lane >> 3, lw = lane & 7;
  const float* src = dense + (((p.n * D + 8LL * p.d) * H + 8LL * p.h + lh) * W + 8LL * p.w + lw) * c;
  const int64_t dstep = H * W * c;  // floats from one d plane to the next
  // The leaf of each voxel of the column.
  int leaf[8], dep[8];
#pragma unroll
  for (int d = 0; d < 8; ++d) {
    const int i = leaf_at(b, d, lh, lw);
    leaf[d] = i;
    dep[d] = i == 0 ? 0 : (i < 9 ? 1 : (i < 73 ? 2 : 3));
  }
  const bool avg = pool == 0;
  for (int k0 = 0; k0 < c; k0 += 4) {
    const int kc = min(4, c - k0);
    // v[d][e]: channel k0 + e of voxel d (0 past c).
    double v[8][4];
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      if constexpr (VEC4) {
        const float4 x = *reinterpret_cast<const float4*>(src + d * dstep + k0);
        v[d][0] = x.x; v[d][1] = x.y; v[d][2] = x.z; v[d][3] = x.w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) v[d][e] = e < kc ? (double)src[d * dstep + k0 + e] : 0.0;
      }
    }
    auto comb = [&](double a, double x) { return avg ? a + x : fmax(a, x); };
    // 2^3 blocks: d pairs, then lanes w ^ 1, h ^ 1 (every lane of the block
    // ends up with the block's value); then 4^3 and 8^3 alike.
    double s2[4][4], s4[2][4], s8[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        double x = comb(v[2 * q][e], v[2 * q + 1][e]);
        x = comb(x, __shfl_xor(x, 1, 64));
        x = comb(x, __shfl_xor(x, 8, 64));
        s2[q][e] = x;
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        double x = comb(s2[2 * q][e], s2[2 * q + 1][e]);
        x = comb(x, __shfl_xor(x, 2, 64));
        x = comb(x, __shfl_xor(x, 16, 64));
        s4[q][e] = x;
      }
      double x = comb(s4[0][e], s4[1][e]);
      x = comb(x, __shfl_xor(x, 4, 64));
      x = comb(x, __shfl_xor(x, 32, 64));
      s8[e] = x;
    }
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      const int dp = dep[d];
      // Cell edge 8 >> depth; this lane writes if the voxel is the cell's first.
      const int msk = (8 >> dp) - 1;
      if ((d & msk) || (lh & msk) || (lw & msk)) continue;
      const int64_t row = row0 + data_idx(b, leaf[d]);
      const double scale = avg ? 1.0 / (double)((8 >> dp) * (8 >> dp) * (8 >> dp)) : 1.0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e >= kc) continue;
        const double x = dp == 3 ? v[d][e] : (dp == 2 ? s2[d >> 1][e] : (dp == 1 ? s4[d >> 2][e] : s8[e]));
        data[row * c + k0 + e] = (float)(avg ? x * scale : x);
      }
    }
  }
}

// W consecutive floats of a row, held as an array so that each component can
// be handled on its own.
template <int W> struct Vec { float v[W]; };

template <int W>
__device__ __forceinline__ Vec<W> vload(const float* __restrict__ p) {
  Vec<W> r;
  if constexpr (W == 4) {
    const float4 x = *reinterpret_cast<const float4*>(p);
    r.v[0] = x.x; r.v[1] = x.y; r.v[2] = x.z; r.v[3] = x.w;
  } else {
    r.v[0] = *p;
  }
  return r;
}

template <int W>
__device__ __forceinline__ void vstore(float* __restrict__ p, const Vec<W>& r) {
  if constexpr (W == 4) *reinterpret_cast<float4*>(p) = make_float4(r.v[0], r.v[1], r.v[2], r.v[3]);
  else *p = r.v[0];
}

// What slots_flush does with one leaf (dst, src, nm), nm being 1 or 8:
//   kRowMax:    out[dst] = max over k < nm of in[src + k] (pooling; nm = 1 copies)
//   kRowSum:    out[dst] = in[src] + in[src + 1] + ... in that order (unpooling
//               gradient; nm = 1 copies)
//   kRowCopy:   out[dst] = in[src] (nm must be 1)
//   kRowArgmax: dst is an output row and src the first of its nm input rows:
//               out[src + k] = in[dst] where x[src + k] is the first maximum
//               of x[src .. src + nm - 1] (per channel), else 0 (pooling gradient)
enum RowOp { kRowMax, kRowSum, kRowCopy, kRowArgmax };

// Pending leaves of a wave in LDS: up to kSlotCap (dst, src, nm) triples.
// Leaves are added a 64-position chunk at a time and handled once 64 or
// more are pending (and at the end), so that a copy phase covers the leaves
// of several chunks and trees.
constexpr int kSlotCap = 128;

struct Slots {
  int64_t* s;
  int count;  // wave-uniform
};

// Adds the leaves marked in m (lane j of m holds dst, src, nm).
__device__ __forceinline__ void slots_add(Slots& sl, uint64_t m, int64_t dst, int64_t src, int nm) {
  const int lane = lane_id();
  if ((m >> lane) & 1ull) {
    const int k = sl.count + __popcll(m & lanemask_lt());
    sl.s[3 * k] = dst;
    sl.s[3 * k + 1] = src;
    sl.s[3 * k + 2] = nm;
  }
  sl.count += __popcll(m);
}

// The row operation on every pending leaf, W floats per lane with several
// leaves side by side (16 leaves per instruction for 16 channels and W = 4).
template <int W, int OP>
__device__ __forceinline__ void slots_flush(Slots& sl, const float* __restrict__ in,
                                            const float* __restrict__ x, int c, float* __restrict__ out) {
  const int nl = sl.count;
  if (nl == 0) return;
  const int64_t* slots = sl.s;
  const int lane = lane_id();
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  const int ne = c / W;
  const int lpr = ne < 64 ? ne : 64;
  const int rpi = 64 / lpr;
  const int q0 = lane % lpr, rsub = lane / lpr;
  for (int r0 = 0; r0 < nl; r0 += rpi) {
    const int r = r0 + rsub;
    if (rsub < rpi && r < nl) {
      const int64_t d = slots[3 * r], sr = slots[3 * r + 1];
      const bool one = slots[3 * r + 2] == 1;
      for (int q = q0; q < ne; q += lpr) {
        const int64_t e = (int64_t)q * W;
        if constexpr (OP == kRowArgmax) {
          const Vec<W> g = vload<W>(in + d * c + e);
          if (one) {
            vstore<W>(out + sr * c + e, g);
            continue;
          }
          Vec<W> xs[8];
#pragma unroll
          for (int k = 0; k < 8; ++k) xs[k] = vload<W>(x + (sr + k) * c + e);
          int arg[W];
          float best[W];
#pragma unroll
          for (int j = 0; j < W; ++j) {
            best[j] = xs[0].v[j];
            arg[j] = 0;
          }
#pragma unroll
          for (int k = 1; k < 8; ++k)
#pragma unroll
            for (int j = 0; j < W; ++j)
              if (xs[k].v[j] > best[j]) {
                best[j] = xs[k].v[j];
                arg[j] = k;
              }
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            Vec<W> o;
#pragma unroll
            for (int j = 0; j < W; ++j) o.v[j] = arg[j] == k ? g.v[j] : 0.f;
            vstore<W>(out + (sr + k) * c + e, o);
          }
        } else {
          Vec<W> v = vload<W>(in + sr * c + e);
          if (OP != kRowCopy && !one) {
            Vec<W> u[7];
#pragma unroll
            for (int k = 0; k < 7; ++k) u[k] = vload<W>(in + (sr + 1 + k) * c + e);
#pragma unroll
            for (int k = 0; k < 7; ++k)
#pragma unroll
              for (int j = 0; j < W; ++j)
                v.v[j] = OP == kRowMax ? fmaxf(v.v[j], u[k].v[j]) : v.v[j] + u[k].v[j];
          }
          vstore<W>(out + d * c + e, v);
        }
      }
    }
  }
  __builtin_amdgcn_wave_barrier();  // the slots are rewritten after this
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  sl.count = 0;
}

// Adds the leaves marked in m and runs the pending ones once 64 or more wait
// (at most 63 + 64 < kSlotCap are then held).
template <int W, int OP>
__device__ __forceinline__ void slots_push(Slots& sl, uint64_t m, int64_t dst, int64_t src, int nm,
                                           const float* __restrict__ in, const float* __restrict__ x,
                                           int c, float* __restrict__ out) {
  slots_add(sl, m, dst, src, nm);
  if (sl.count >= 64) slots_flush<W, OP>(sl, in, x, c, out);
}

// Eq. 10 data: one wave per output tree.
template <int W>
__global__ void __launch_bounds__(256) k_pool_max(const uint32_t* __restrict__ in_trees,
                                                  const int64_t* __restrict__ in_prefix, int64_t n_out,
                                                  int gd, int gh, int gw, const float* __restrict__ in,
                                                  int c, const uint32_t* __restrict__ out_trees,
                                                  const int64_t* __restrict__ out_prefix,
                                                  float* __restrict__ out) {
  __shared__ int64_t slots_all[4][3 * kSlotCap];
  Slots sl{slots_all[threadIdx.x >> 6], 0};
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_out) return;
  const TreePos p = tree_pos(t, gd / 2, gh / 2, gw / 2);
  const Bits ob = load_bits(out_trees, t);
  const int64_t row0 = out_prefix[t];
  int base = 0;
  // No split depth-2 node: no leaf past position 72.
  const int nend = (((ob.lo >> 9) != 0ull) || ob.hi) ? kNodes : 73;
  for (int c0 = 0; c0 < nend; c0 += 64) {
    const int i = c0 + lane_id();
    const bool leaf = i < kNodes && is_leaf(ob, i);
    const uint64_t m = __ballot(leaf);
    int64_t orow = 0, srow = 0;
    int nmax = 1;
    if (leaf) {
      orow = row0 + base + __popcll(m & lanemask_lt());
      int o, node;
      if (i < 9) {          // output depth 1 <- input root
        o = i - 1; node = 0;
      } else if (i < 73) {  // output depth 2 <- input depth 1
        o = (i - 9) >> 3; node = 1 + ((i - 9) & 7);
      } else {              // output depth 3 <- input depth 2 node
        o = (i - 73) >> 6; node = 9 + ((i - 73) & 63);
      }
      const int64_t ti = ((p.n * gd + 2 * p.d + ((o >> 2) & 1)) * gh + 2 * p.h + ((o >> 1) & 1)) * gw +
                         2 * p.w + (o & 1);
      const Bits ib = load_bits(in_trees, ti);
      if (node >= 9 && bit(ib, node)) {  // split depth-2 node: max of its 8 voxels
        node = 8 * node + 1;
        nmax = 8;
      }
      srow = in_prefix[ti] + data_idx(ib, node);
    }
    slots_push<W, kRowMax>(sl, m, orow, srow, nmax, in, nullptr, c, out);
    base += __popcll(m);
  }
  slots_flush<W, kRowMax>(sl, in, nullptr, c, out);
}

// Eq. 12 data (plain or guided): one wave per input tree and its 8 output
// trees.  An output tree with a single leaf copies the input leaf that holds
// it (the input node 1 + o, or the input root when that is unsplit); the
// leaves of a split output tree are enumerated 64 positions at a time and
// each copies the input leaf holding its voxels at half resolution.
template <int W>
__global__ void __launch_bounds__(256) k_unpool(const uint32_t* __restrict__ in_trees,
                                                const int64_t* __restrict__ in_prefix, int64_t n_in,
                                                int gd, int gh, int gw, const float* __restrict__ in,
                                                int c, const uint32_t* __restrict__ out_trees,
                                                const int64_t* __restrict__ out_prefix,
                                                float* __restrict__ out) {
  __shared__ int64_t slots_all[4][3 * kSlotCap];
  const int wave = threadIdx.x >> 6;
  const int64_t ti = (int64_t)blockIdx.x * 4 + wave;
  if (ti >= n_in) return;  // whole wave exits together
  Slots sl{slots_all[wave], 0};
  const int lane = lane_id();
  const TreePos p = tree_pos(ti, gd, gh, gw);
  const Bits ib = load_bits(in_trees, ti);
  const int64_t in_row0 = in_prefix[ti];
  const bool in_split = (ib.lo & 1ull) != 0;
  const int Gh = 2 * gh, Gw = 2 * gw, Gd = 2 * gd;
  // Lane o < 8 loads output tree o's bits and first row; split trees take
  // them from that lane.
  bool single = false;
  Bits obl{0ull, 0u};
  int64_t orow = 0, srow = 0;
  if (lane < 8) {
    const int o = lane;
    const int64_t t = ((p.n * Gd + 2 * p.d + ((o >> 2) & 1)) * Gh + 2 * p.h + ((o >> 1) & 1)) * Gw +
                      2 * p.w + (o & 1);
    obl = load_bits(out_trees, t);
    single = !(obl.lo & 1ull);
    orow = out_prefix[t];
    srow = in_row0 + data_idx(ib, in_split ? 1 + lane : 0);
  }
  const uint64_t singles = __ballot(single);
  const uint64_t split = __ballot(lane < 8 && !single);
  // Output trees with a single leaf.
  slots_add(sl, singles, orow, srow, 1);
  // Split output trees.
  for (uint32_t sm = (uint32_t)split; sm; sm &= sm - 1) {
    const int o = __ffs(sm) - 1;
    Bits ob;
    ob.lo = __shfl(obl.lo, o, 64);
    ob.hi = __shfl(obl.hi, o, 64);
    const int64_t row0 = __shfl(orow, o, 64);
    int base = 0;
    // No split depth-2 node: no leaf past position 72.
    const int nend = (((ob.lo >> 9) != 0ull) || ob.hi) ? kNodes : 73;
    for (int c0 = 1; c0 < nend; c0 += 64) {
      const int i = c0 + lane;
      const bool leaf = i < kNodes && is_leaf(ob, i);
      const uint64_t m = __ballot(leaf);
      int64_t lo = 0, ls = 0;
      if (leaf) {
        lo = row0 + base + __popcll(m & lanemask_lt());
        int node;
        if (!in_split) node = 0;                       // unsplit input tree (guided only)
        else if (i < 9) node = 9 + 8 * o + (i - 1);    // depth 1 <- depth 2
        else if (i < 73) node = 73 + 64 * o + (i - 9); // depth 2 <- depth-3 voxel
        else node = 73 + 64 * o + ((i - 73) >> 3);     // guided depth 3 <- same voxel
        ls = in_row0 + data_idx(ib, node);
      }
      slots_push<W, kRowCopy>(sl, m, lo, ls, 1, in, nullptr, c, out);
      base += __popcll(m);
    }
  }
  slots_flush<W, kRowCopy>(sl, in, nullptr, c, out);
}

__global__ void k_relu(float* __restrict__ x, int64_t count) {
  const int64_t n4 = count >> 2;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  float4* x4 = reinterpret_cast<float4*>(x);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 v = x4[i];
    v.x = fmaxf(v.x, 0.f); v.y = fmaxf(v.y, 0.f); v.z = fmaxf(v.z, 0.f); v.w = fmaxf(v.w, 0.f);
    x4[i] = v;
  }
  for (int64_t i = 4 * n4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride)
    x[i] = fmaxf(x[i], 0.f);
}

__global__ void k_relu_scalar(float* __restrict__ x, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride)
    x[i] = fmaxf(x[i], 0.f);
}

// ---------------------------------------------------------------------------
// Gradients of pooling, unpooling and ReLU.
// ---------------------------------------------------------------------------

// Gradient of Eq. 10: an output leaf that copies one input leaf passes dy to
// it; one that takes the maximum of 8 unit voxels passes dy, per channel, to
// the first voxel (in child order) holding the maximum and 0 to the others.
// Every input leaf has exactly one output leaf, so every row of din is
// written once.  One wave per output tree, as the forward kernel.
template <int W>
__global__ void __launch_bounds__(256) k_pool_max_bwd(
    const uint32_t* __restrict__ in_trees, const int64_t* __restrict__ in_prefix, int64_t n_out,
    int gd, int gh, int gw, const float* __restrict__ in, int c,
    const uint32_t* __restrict__ out_trees, const int64_t* __restrict__ out_prefix,
    const float* __restrict__ dy, float* __restrict__ din) {
  __shared__ int64_t slots_all[4][3 * kSlotCap];
  Slots sl{slots_all[threadIdx.x >> 6], 0};
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_out) return;
  const TreePos p = tree_pos(t, gd / 2, gh / 2, gw / 2);
  const Bits ob = load_bits(out_trees, t);
  const int64_t row0 = out_prefix[t];
  int base = 0;
  // No split depth-2 node: no leaf past position 72.
  const int nend = (((ob.lo >> 9) != 0ull) || ob.hi) ? kNodes : 73;
  for (int c0 = 0; c0 < nend; c0 += 64) {
    const int i = c0 + lane_id();
    const bool leaf = i < kNodes && is_leaf(ob, i);
    const uint64_t m = __ballot(leaf);
    int64_t orow = 0, srow = 0;
    int nmax = 1;
    if (leaf) {
      orow = row0 + base + __popcll(m & lanemask_lt());
      int o, node;
      if (i < 9) {
        o = i - 1; node = 0;
      } else if (i < 73) {
        o = (i - 9) >> 3; node = 1 + ((i - 9) & 7);
      } else {
        o = (i - 73) >> 6; node = 9 + ((i - 73) & 63);
      }
      const int64_t ti = ((p.n * gd + 2 * p.d + ((o >> 2) & 1)) * gh + 2 * p.h + ((o >> 1) & 1)) * gw +
                         2 * p.w + (o & 1);
      const Bits ib = load_bits(in_trees, ti);
      if (node >= 9 && bit(ib, node)) {
        node = 8 * node + 1;
        nmax = 8;
      }
      srow = in_prefix[ti] + data_idx(ib, node);
    }
    slots_push<W, kRowArgmax>(sl, m, orow, srow, nmax, dy, in, c, din);
    base += __popcll(m);
  }
  slots_flush<W, kRowArgmax>(sl, dy, in, c, din);
}

// Gradient of Eq. 12 (plain or guided): every input leaf receives the sum of
// dy over the output leaves that copy it, in output row order.  One wave per
// input tree, as the forward kernel; each input leaf is written once, from
// what it gathers:
//   - an unsplit input root: the 8 single-leaf output trees it spawned;
//   - an output tree with a single leaf: that row (input node 1 + o);
//   - in a split output tree, a leaf above depth 3: its own row (input leaf
//     one level deeper); the 8 depth-3 leaves of a split depth-2 node (guided
//     only): their 8 consecutive rows, summed into the input voxel that
//     pooled them.
// The output structure is the plain unpooling of the input or a guide that
// pools to it, so every input leaf is covered.
template <int W>
__global__ void __launch_bounds__(256) k_unpool_bwd(
    const uint32_t* __restrict__ in_trees, const int64_t* __restrict__ in_prefix, int64_t n_in,
    int gd, int gh, int gw, int c, const uint32_t* __restrict__ out_trees,
    const int64_t* __restrict__ out_prefix, const float* __restrict__ dy, float* __restrict__ din) {
  __shared__ int64_t slots_all[4][3 * kSlotCap];
  const int wave = threadIdx.x >> 6;
  const int64_t ti = (int64_t)blockIdx.x * 4 + wave;
  if (ti >= n_in) return;  // whole wave exits together
  Slots sl{slots_all[wave], 0};
  const int lane = lane_id();
  const TreePos p = tree_pos(ti, gd, gh, gw);
  const Bits ib = load_bits(in_trees, ti);
  const int64_t in_row0 = in_prefix[ti];
  const bool in_split = (ib.lo & 1ull) != 0;
  const int Gh = 2 * gh, Gw = 2 * gw, Gd = 2 * gd;
  // Lane o < 8 loads output tree o's bits and first row.
  bool single = false;
  Bits obl{0ull, 0u};
  int64_t orow = 0, irow = 0;
  if (lane < 8) {
    const int o = lane;
    const int64_t t = ((p.n * Gd + 2 * p.d + ((o >> 2) & 1)) * Gh + 2 * p.h + ((o >> 1) & 1)) * Gw +
                      2 * p.w + (o & 1);
    obl = load_bits(out_trees, t);
    single = !(obl.lo & 1ull);
    orow = out_prefix[t];
    irow = in_row0 + (in_split ? data_idx(ib, 1 + lane) : 0);
  }
  if (!in_split) {
    int64_t r[8];
#pragma unroll
    for (int o = 0; o < 8; ++o) r[o] = __shfl(orow, o, 64);
    const int ne = c / W;
    for (int q = lane; q < ne; q += 64) {
      const int64_t e = (int64_t)q * W;
      Vec<W> v = vload<W>(dy + r[0] * c + e);
      Vec<W> u[7];
#pragma unroll
      for (int o = 0; o < 7; ++o) u[o] = vload<W>(dy + r[o + 1] * c + e);
#pragma unroll
      for (int o = 0; o < 7; ++o)
#pragma unroll
        for (int j = 0; j < W; ++j) v.v[j] += u[o].v[j];
      vstore<W>(din + in_row0 * c + e, v);
    }
    return;
  }
  const uint64_t singles = __ballot(lane < 8 && single);
  const uint64_t split = __ballot(lane < 8 && !single);
  slots_add(sl, singles, irow, orow, 1);
  for (uint32_t sm = (uint32_t)split; sm; sm &= sm - 1) {
    const int o = __ffs(sm) - 1;
    Bits ob;
    ob.lo = __shfl(obl.lo, o, 64);
    ob.hi = __shfl(obl.hi, o, 64);
    const int64_t row0 = __shfl(orow, o, 64);
    int base = 0;
    // No split depth-2 node: no leaf past position 72.
    const int nend = (((ob.lo >> 9) != 0ull) || ob.hi) ? kNodes : 73;
    for (int c0 = 1; c0 < nend; c0 += 64) {
      const int i = c0 + lane;
      const bool leaf = i < kNodes && is_leaf(ob, i);
      const uint64_t m = __ballot(leaf);
      // Depth-3 leaves come as 8 siblings in consecutive rows (inside one
      // 64-position chunk, as 73 + 8k and the chunk starts are 8-aligned
      // relative to each other); the first one stands for all 8.
      const bool head = leaf && (i < 73 || ((i - 73) & 7) == 0);
      const uint64_t h = __ballot(head);
      int64_t dst = 0, src = 0;
      int nm = 1;
      if (head) {
        src = row0 + base + __popcll(m & lanemask_lt());
        int node;
        if (i < 9) {
          node = 9 + 8 * o + (i - 1);        // depth 1 <- depth 2
        } else if (i < 73) {
          node = 73 + 64 * o + (i - 9);      // depth 2 <- depth-3 voxel
        } else {
          node = 73 + 64 * o + ((i - 73) >> 3);  // guided depth 3 <- same voxel
          nm = 8;
        }
        dst = in_row0 + data_idx(ib, node);
      }
      slots_push<W, kRowSum>(sl, h, dst, src, nm, dy, nullptr, c, din);
      base += __popcll(m);
    }
  }
  slots_flush<W, kRowSum>(sl, dy, nullptr, c, din);
}

// Channel concatenation of two leaf arrays on one structure (the skip
// connections of the encoder-decoder): out[row] = [a[row], b[row]], and its
// gradient, the split of dout into da and db (either may be null).  V floats
// per thread (ca, cb divisible by V).
template <int V>
__global__ void k_concat(const float* __restrict__ a, int ca, const float* __restrict__ b, int cb,
                         int64_t n_rows, float* __restrict__ out) {
  typedef typename VecF<V>::type T;
  const int va = ca / V, vc = (ca + cb) / V;
  const int64_t n = n_rows * vc;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int64_t row = i / vc;
    const int k = (int)(i - row * vc);
    reinterpret_cast<T*>(out)[i] = k < va ? reinterpret_cast<const T*>(a)[row * va + k]
                                          : reinterpret_cast<const T*>(b)[row * (vc - va) + (k - va)];
  }
}

template <int V>
__global__ void k_split(const float* __restrict__ dout, int ca, int cb, int64_t n_rows,
                        float* __restrict__ da, float* __restrict__ db) {
  typedef typename VecF<V>::type T;
  const int va = ca / V, vc = (ca + cb) / V;
  const int64_t n = n_rows * vc;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int64_t row = i / vc;
    const int k = (int)(i - row * vc);
    const T v = reinterpret_cast<const T*>(dout)[i];
    if (k < va) {
      if (da) reinterpret_cast<T*>(da)[row * va + k] = v;
    } else if (db) {
      reinterpret_cast<T*>(db)[row * (vc - va) + (k - va)] = v;
    }
  }
}

// out = a + b on leaf data (gradient accumulation where a layer output
// feeds two layers, as an encoder output feeding both the next level and a
// concat).  out may alias a or b.
__global__ void k_add(const float* a, const float* b, float* out, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride)
    out[i] = a[i] + b[i];
}

// din = dy where the ReLU output y is positive, else 0.  din may alias dy.
__global__ void k_relu_bwd(const float* y, const float* dy, float* din, int64_t count) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride)
    din[i] = y[i] > 0.f ? dy[i] : 0.f;
}

}  // namespace

namespace oci {

hipError_t launch_oc2ten(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
                         int gw, const float* data, int c, float* dense, hipStream_t s) {
  const int64_t nv = 512LL * n * gd * gh * gw;
  hipLaunchKernelGGL(k_oc2ten, dim3(blocks_for(nv, 256)), dim3(256), 0, s, trees, prefix, nv, gd,
                     gh, gw, data, c, dense);
  return hipGetLastError();
}

hipError_t launch_ten2oc(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
                         int gw, const float* dense, int c, int pool, float* data, hipStream_t s) {
  const int64_t nt = (int64_t)n * gd * gh * gw;
  if (c % 4 == 0 && (reinterpret_cast<uintptr_t>(dense) & 15) == 0)
    hipLaunchKernelGGL(k_ten2oc<true>, dim3(blocks_for(nt, 4)), dim3(256), 0, s, trees, prefix, nt, gd, gh,
                       gw, dense, c, pool, data);
  else
    hipLaunchKernelGGL(k_ten2oc<false>, dim3(blocks_for(nt, 4)), dim3(256), 0, s, trees, prefix, nt, gd, gh,
                       gw, dense, c, pool, data);
  return hipGetLastError();
}

hipError_t launch_pool_max(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd,
                           int gh, int gw, const float* in, int c, const uint32_t* out_trees,
                           const int64_t* out_prefix, float* out, hipStream_t s) {
  const int64_t no = (int64_t)n * (gd / 2) * (gh / 2) * (gw / 2);
  const bool vec = c % 4 == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(k_pool_max<4>, dim3(blocks_for(no, 4)), dim3(256), 0, s, in_trees, in_prefix, no,
                       gd, gh, gw, in, c, out_trees, out_prefix, out);
  else
    hipLaunchKernelGGL(k_pool_max<1>, dim3(blocks_for(no, 4)), dim3(256), 0, s, in_trees, in_prefix, no,
                       gd, gh, gw, in, c, out_trees, out_prefix, out);
  return hipGetLastError();
}

hipError_t launch_unpool(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh,
                         int gw, const float* in, int c, const uint32_t* out_trees,
                         const int64_t* out_prefix, float* out, hipStream_t s) {
  const int64_t ni = (int64_t)n * gd * gh * gw;
  const bool vec = c % 4 == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(out) & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(k_unpool<4>, dim3(blocks_for(ni, 4)), dim3(256), 0, s, in_trees, in_prefix, ni,
                       gd, gh, gw, in, c, out_trees, out_prefix, out);
  else
    hipLaunchKernelGGL(k_unpool<1>, dim3(blocks_for(ni, 4)), dim3(256), 0, s, in_trees, in_prefix, ni,
                       gd, gh, gw, in, c, out_trees, out_prefix, out);
  return hipGetLastError();
}

hipError_t launch_relu(float* x, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  int64_t blocks = (count / 4 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  if ((reinterpret_cast<uintptr_t>(x) & 15) != 0) {  // float4 path needs 16-byte alignment
    hipLaunchKernelGGL(k_relu_scalar, dim3((unsigned)blocks), dim3(256), 0, s, x, count);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_relu, dim3((unsigned)blocks), dim3(256), 0, s, x, count);
  return hipGetLastError();
}

hipError_t launch_pool_max_bwd(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd,
                               int gh, int gw, const float* in, int c, const uint32_t* out_trees,
                               const int64_t* out_prefix, const float* dy, float* din,
                               hipStream_t s) {
  const int64_t no = (int64_t)n * (gd / 2) * (gh / 2) * (gw / 2);
  const bool vec = c % 4 == 0 && (reinterpret_cast<uintptr_t>(in) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(dy) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(din) & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(k_pool_max_bwd<4>, dim3(blocks_for(no, 4)), dim3(256), 0, s, in_trees, in_prefix,
                       no, gd, gh, gw, in, c, out_trees, out_prefix, dy, din);
  else
    hipLaunchKernelGGL(k_pool_max_bwd<1>, dim3(blocks_for(no, 4)), dim3(256), 0, s, in_trees, in_prefix,
                       no, gd, gh, gw, in, c, out_trees, out_prefix, dy, din);
  return hipGetLastError();
}

hipError_t launch_unpool_bwd(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd,
                             int gh, int gw, int64_t in_n_leaves, int c, const uint32_t* out_trees,
                             const int64_t* out_prefix, const float* dy, float* din,
                             hipStream_t s) {
  (void)in_n_leaves;  // every input row is written by the gather
  const int64_t ni = (int64_t)n * gd * gh * gw;
  const bool vec = c % 4 == 0 && (reinterpret_cast<uintptr_t>(dy) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(din) & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(k_unpool_bwd<4>, dim3(blocks_for(ni, 4)), dim3(256), 0, s, in_trees, in_prefix, ni,
                       gd, gh, gw, c, out_trees, out_prefix, dy, din);
  else
    hipLaunchKernelGGL(k_unpool_bwd<1>, dim3(blocks_for(ni, 4)), dim3(256), 0, s, in_trees, in_prefix, ni,
                       gd, gh, gw, c, out_trees, out_prefix, dy, din);
  return hipGetLastError();
}

hipError_t launch_relu_bwd(const float* y, const float* dy, float* din, int64_t count,
                           hipStream_t s) {
  if (count <= 0) return hipSuccess;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_relu_bwd, dim3((unsigned)blocks), dim3(256), 0, s, y, dy, din, count);
  return hipGetLastError();
}

hipError_t launch_concat(const float* a, int ca, const float* b, int cb, int64_t n_rows, float* out,
                         hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  const uintptr_t al = reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b) |
                       reinterpret_cast<uintptr_t>(out);
  const bool v4 = ca % 4 == 0 && cb % 4 == 0 && (al & 15) == 0;
  const int64_t n = n_rows * (int64_t)(ca + cb) / (v4 ? 4 : 1);
  int64_t blocks = (n + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  if (v4)
    hipLaunchKernelGGL(k_concat<4>, dim3((unsigned)blocks), dim3(256), 0, s, a, ca, b, cb, n_rows, out);
  else
    hipLaunchKernelGGL(k_concat<1>, dim3((unsigned)blocks), dim3(256), 0, s, a, ca, b, cb, n_rows, out);
  return hipGetLastError();
}

hipError_t launch_split(const float* dout, int ca, int cb, int64_t n_rows, float* da, float* db,
                        hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  const uintptr_t al = reinterpret_cast<uintptr_t>(dout) | reinterpret_cast<uintptr_t>(da) |
                       reinterpret_cast<uintptr_t>(db);
  const bool v4 = ca % 4 == 0 && cb % 4 == 0 && (al & 15) == 0;
  const int64_t n = n_rows * (int64_t)(ca + cb) / (v4 ? 4 : 1);
  int64_t blocks = (n + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  if (v4)
    hipLaunchKernelGGL(k_split<4>, dim3((unsigned)blocks), dim3(256), 0, s, dout, ca, cb, n_rows, da, db);
  else
    hipLaunchKernelGGL(k_split<1>, dim3((unsigned)blocks), dim3(256), 0, s, dout, ca, cb, n_rows, da, db);
  return hipGetLastError();
}

hipError_t launch_add(const float* a, const float* b, float* out, int64_t count, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  hipLaunchKernelGGL(k_add, dim3((unsigned)blocks), dim3(256), 0, s, a, b, out, count);
  return hipGetLastError();
}

}  // namespace oci
