// Structure kernels: octree build, leaf counts and prefix scan, leaf index,
// voxel->row map, canonical-form check, and the structure side of 2x2x2
// pooling / unpooling (OctNet Sec. 3.1, Eq. 1-3, Eq. 10, Eq. 12).
#include <type_traits>

#include "oc_internal.h"

using namespace ocd;

namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanChunk = kScanThreads * kScanItems;

// ---------------------------------------------------------------------------
// Build.  A workgroup takes up to kBuildTrees consecutive trees along w (one
// row of the same n, d, h): their 64 voxel rows of 8 bytes each are
// contiguous per row (256 bytes for 32 trees), so the rows are read as whole
// cache lines into LDS, 16 bytes per lane where the grid width is even.
// The any-occupied / all-occupied flags of the 64 depth-2 blocks (2x2x2
// voxels, node q = 8 o1 + o2 at bit 9 + q) of a tree then give every split
// decision of the tree.
// ---------------------------------------------------------------------------
constexpr int kBuildTrees = 32;
#ifndef OC_BUILD_THREADS
#define OC_BUILD_THREADS 256
#endif
#ifndef OC_BUILD_SEGS
#define OC_BUILD_SEGS 1
#endif
constexpr int kBuildThreads = OC_BUILD_THREADS;
constexpr int kBuildSegs = OC_BUILD_SEGS;       // segments of up to 32 trees per workgroup
constexpr int kBuildStride = kBuildTrees + 1;  // uint2 per LDS row (padding against bank conflicts)

// Segment seg of the grid: trees [tw0, tw0 + count) of line (n, tree d, tree h).
struct BuildSeg {
  int64_t line;
  int tw0, count;
};

__device__ __forceinline__ BuildSeg build_seg(int64_t seg, int64_t n_lines, int gw) {
  const int wblocks = (gw + kBuildTrees - 1) / kBuildTrees;
  BuildSeg b;
  b.line = seg / wblocks;
  b.tw0 = kBuildTrees * (int)(seg % wblocks);
  b.count = b.line < n_lines ? min(kBuildTrees, gw - b.tw0) : 0;
  return b;
}

template <bool PAIRS>
__global__ void __launch_bounds__(kBuildThreads) k_build(const uint8_t* __restrict__ occ, int64_t n_trees,
                                                        int gd, int gh, int gw, int rule,
                                                        uint32_t* __restrict__ trees,
                                                        int32_t* __restrict__ counts) {
  __shared__ uint2 rows[kBuildSegs][64 * kBuildStride];  // [seg][voxel row 8 d + h][tree] 8 voxels along w
  const int64_t n_lines = n_trees / gw;
  const int64_t H = 8LL * gh, W = 8LL * gw, D = 8LL * gd;
  // Every segment's row pieces are loaded before any is stored.
  constexpr int PER = PAIRS ? kBuildTrees / 2 : kBuildTrees;  // loads per voxel row
  constexpr int NL = 64 * PER / kBuildThreads;
  using V = typename std::conditional<PAIRS, uint4, uint2>::type;
  V v[kBuildSegs][NL];
#pragma unroll
  for (int sg = 0; sg < kBuildSegs; ++sg) {
    const BuildSeg b = build_seg((int64_t)blockIdx.x * kBuildSegs + sg, n_lines, gw);
    const int th = (int)(b.line % gh);
    const int td = (int)((b.line / gh) % gd);
    const int64_t n = b.line / ((int64_t)gh * gd);
    const uint8_t* base = occ + ((n * D + 8LL * td) * H + 8LL * th) * W + 8LL * b.tw0;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int k = threadIdx.x + kBuildThreads * i;
      const int r = k / PER, tl = (PAIRS ? 2 : 1) * (k % PER);  // r = 8 d + h
      if constexpr (PAIRS) v[sg][i] = make_uint4(0u, 0u, 0u, 0u);
      else v[sg][i] = make_uint2(0u, 0u);
      // PAIRS: count is even (gw and kBuildTrees are)
      if (tl < b.count) v[sg][i] = *reinterpret_cast<const V*>(base + ((r >> 3) * H + (r & 7)) * W + 8 * tl);
    }
  }
#pragma unroll
  for (int sg = 0; sg < kBuildSegs; ++sg)
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int k = threadIdx.x + kBuildThreads * i;
      const int r = k / PER, tl = (PAIRS ? 2 : 1) * (k % PER);
      if constexpr (PAIRS) {
        rows[sg][r * kBuildStride + tl] = make_uint2(v[sg][i].x, v[sg][i].y);
        rows[sg][r * kBuildStride + tl + 1] = make_uint2(v[sg][i].z, v[sg][i].w);
      } else {
        rows[sg][r * kBuildStride + tl] = v[sg][i];
      }
    }
  __syncthreads();
  // Then 16 lanes per tree, 4 trees per wave: lane (dp, hp) takes the voxel
  // rows d = 2 dp + {0, 1}, h = 2 hp + {0, 1} of its tree, i.e. the four
  // depth-2 blocks w = 2j + {0, 1} (j = 0..3) there, and finds for each
  // whether any / all of its 8 voxels are occupied; OR over the tree's 16
  // lanes gives the 64-bit any / all masks by depth-2 node q = 8 o1 + o2.
  const int lane = lane_id();
  const int grp = lane >> 4, dp = (lane >> 2) & 3, hp = lane & 3;
  constexpr uint64_t kLow = 0x0101010101010101ull;
  for (int sg = 0; sg < kBuildSegs; ++sg) {
    const BuildSeg b = build_seg((int64_t)blockIdx.x * kBuildSegs + sg, n_lines, gw);
    for (int tl0 = (threadIdx.x >> 6) * 4; tl0 < b.count; tl0 += kBuildThreads / 16) {
      const int tl = tl0 + grp;
      uint64_t any8 = 0, all8 = kLow;  // per voxel column: some / every row occupied
      if (tl < b.count) {
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const uint2 r2 = rows[sg][((2 * dp + a) * 8 + 2 * hp + c) * kBuildStride + tl];
            uint64_t t = (uint64_t)r2.x | ((uint64_t)r2.y << 32);
            t |= (t >> 4) & 0x0F0F0F0F0F0F0F0Full;
            t |= (t >> 2) & 0x3333333333333333ull;
            t |= (t >> 1) & 0x5555555555555555ull;
            t &= kLow;  // bit 8k: voxel k of the row is occupied
            any8 |= t;
            all8 &= t;
          }
      }
      uint64_t A = 0, L = 0;
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) {
        const uint32_t an = (uint32_t)(any8 >> (16 * jb)) & 0x0101u;
        const uint32_t al = (uint32_t)(all8 >> (16 * jb)) & 0x0101u;
        const int o1 = 4 * (dp >> 1) + 2 * (hp >> 1) + (jb >> 1);
        const int o2 = 4 * (dp & 1) + 2 * (hp & 1) + (jb & 1);
        const int qb = 8 * o1 + o2;
        A |= (uint64_t)(an != 0u) << qb;
        L |= (uint64_t)(al == 0x0101u) << qb;
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        A |= __shfl_xor(A, off, 64);
        L |= __shfl_xor(L, off, 64);
      }
      const uint64_t split2_ok = rule == 0 ? (A & ~L) : A;
      const int split0 = rule == 0 ? (A != 0ull && L != ~0ull) : (A != 0ull);
      uint32_t s1 = 0;
      uint64_t s2 = 0;
      if (split0) {
#pragma unroll
        for (int o = 0; o < 8; ++o) {
          const uint32_t ga = (uint32_t)((A >> (8 * o)) & 0xFFull);
          const uint32_t gl = (uint32_t)((L >> (8 * o)) & 0xFFull);
          const int sp = rule == 0 ? (ga != 0u && gl != 0xFFu) : (ga != 0u);
          if (sp) {
            s1 |= 1u << o;
            s2 |= split2_ok & (0xFFull << (8 * o));
          }
        }
      }
      if ((lane & 15) == 0 && tl < b.count) {
        const int64_t t = b.line * gw + b.tw0 + tl;
        const uint64_t lo = (uint64_t)split0 | ((uint64_t)s1 << 1) | (s2 << 9);
        const uint32_t hi = (uint32_t)(s2 >> 55);
        uint4 w;
        w.x = (uint32_t)lo;
        w.y = (uint32_t)(lo >> 32);
        w.z = hi;
        w.w = 0u;
        reinterpret_cast<uint4*>(trees)[t] = w;
        counts[t] = 1 + 7 * (split0 + __popc(s1) + __popcll(s2));
      }
    }
  }
}

__global__ void k_count(const uint32_t* __restrict__ trees, int64_t n_trees,
                        int32_t* __restrict__ counts) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_trees) return;
  counts[t] = n_leaves_of(load_bits(trees, t));
}

__global__ void k_validate(const uint32_t* __restrict__ trees, int64_t n_trees,
                           int32_t* __restrict__ n_bad) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_trees) return;
  const uint4 w = reinterpret_cast<const uint4*>(trees)[t];
  int ok = (w.z >> 9) == 0u && w.w == 0u;
  const Bits b = load_bits(trees, t);
  // every set bit i >= 1 needs its parent set
  for (int i = 1; i < kBits && ok; ++i)
    if (bit(b, i) && !bit(b, (i - 1) >> 3)) ok = 0;
  if (!ok) atomicAdd(n_bad, 1);
}

// ---------------------------------------------------------------------------
// Exclusive scan of int32 counts into int64 prefix (three passes).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int64_t wave_incl_scan(int64_t v) {
  const int l = lane_id();
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int64_t u = __shfl_up(v, off, 64);
    if (l >= off) v += u;
  }
  return v;
}

// Exclusive scan of one value per thread over a 256-thread block.
__device__ __forceinline__ int64_t block_excl_scan(int64_t v, int64_t* sh_waves, int64_t* total) {
  const int wv = threadIdx.x >> 6;
  const int64_t incl = wave_incl_scan(v);
  if (lane_id() == 63) sh_waves[wv] = incl;
  __syncthreads();
  int64_t off = 0, tot = 0;
  for (int k = 0; k < (int)(blockDim.x >> 6); ++k) {
    if (k < wv) off += sh_waves[k];
    tot += sh_waves[k];
  }
  __syncthreads();
  *total = tot;
  return off + incl - v;
}

// A thread's kScanItems consecutive counts from base (zero past n): 16-byte
// loads when all are in range and the array is 16-byte aligned.
__device__ __forceinline__ void load_items(const int32_t* __restrict__ counts, int64_t base, int64_t n,
                                           int32_t (&v)[kScanItems]) {
  if (base + kScanItems <= n && (reinterpret_cast<uintptr_t>(counts) & 15) == 0) {
    const int4* q = reinterpret_cast<const int4*>(counts + base);
#pragma unroll
    for (int i = 0; i < kScanItems / 4; ++i) {
      const int4 x = q[i];
      v[4 * i] = x.x;
      v[4 * i + 1] = x.y;
      v[4 * i + 2] = x.z;
      v[4 * i + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) v[k] = base + k < n ? counts[base + k] : 0;
  }
}

// Writes the exclusive prefix run + v[0] + ... + v[k - 1] to prefix[base + k]
// (k < kScanItems, base + k < n): 16-byte stores when all are in range and
// the array is 16-byte aligned.
__device__ __forceinline__ void store_items(int64_t* __restrict__ prefix, int64_t base, int64_t n, int64_t run,
                                            const int32_t (&v)[kScanItems]) {
  int64_t r[kScanItems];
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    r[k] = run;
    run += v[k];
  }
  if (base + kScanItems <= n && (reinterpret_cast<uintptr_t>(prefix) & 15) == 0) {
    longlong2* q = reinterpret_cast<longlong2*>(prefix + base);
#pragma unroll
    for (int i = 0; i < kScanItems / 2; ++i) q[i] = make_longlong2(r[2 * i], r[2 * i + 1]);
  } else {
#pragma unroll
    for (int k = 0; k < kScanItems; ++k)
      if (base + k < n) prefix[base + k] = r[k];
  }
}

// Several scans of the same length at once (blockIdx.y selects the array).
struct ScanSet {
  const int32_t* counts[oci::kMaxScans];
  int64_t* prefix[oci::kMaxScans];
  int64_t* sums[oci::kMaxScans];
};

__global__ void __launch_bounds__(kScanThreads) k_scan_reduce(const int32_t* __restrict__ counts,
                                                              int64_t n, int64_t* __restrict__ sums) {
  __shared__ int64_t sh[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  load_items(counts, base, n, v);
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) s += v[k];
  int64_t tot;
  block_excl_scan(s, sh, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

__global__ void __launch_bounds__(kScanThreads) k_scan_reduce_set(ScanSet set, int64_t n) {
  __shared__ int64_t sh[kScanThreads / 64];
  const int32_t* __restrict__ counts = set.counts[blockIdx.y];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  load_items(counts, base, n, v);
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) s += v[k];
  int64_t tot;
  block_excl_scan(s, sh, &tot);
  if (threadIdx.x == 0) set.sums[blockIdx.y][blockIdx.x] = tot;
}

// Single block: exclusive scan of the per-chunk sums in place; total -> *total.
__global__ void __launch_bounds__(kScanThreads) k_scan_sums(int64_t* __restrict__ sums, int64_t nb,
                                                            int64_t* __restrict__ total) {
  __shared__ int64_t sh[kScanThreads / 64];
  int64_t carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += kScanThreads) {
    const int64_t i = b0 + threadIdx.x;
    const int64_t v = i < nb ? sums[i] : 0;
    int64_t tot;
    const int64_t ex = block_excl_scan(v, sh, &tot);
    if (i < nb) sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) *total = carry;
}

__global__ void __launch_bounds__(kScanThreads) k_scan_sums_set(ScanSet set, int64_t nb, int64_t n) {
  __shared__ int64_t sh[kScanThreads / 64];
  int64_t* __restrict__ sums = set.sums[blockIdx.y];
  int64_t carry = 0;
  for (int64_t b0 = 0; b0 < nb; b0 += kScanThreads) {
    const int64_t i = b0 + threadIdx.x;
    const int64_t v = i < nb ? sums[i] : 0;
    int64_t tot;
    const int64_t ex = block_excl_scan(v, sh, &tot);
    if (i < nb) sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0) set.prefix[blockIdx.y][n] = carry;
}

__global__ void __launch_bounds__(kScanThreads) k_scan_apply_set(ScanSet set, int64_t n) {
  __shared__ int64_t sh[kScanThreads / 64];
  const int32_t* __restrict__ counts = set.counts[blockIdx.y];
  int64_t* __restrict__ prefix = set.prefix[blockIdx.y];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  load_items(counts, base, n, v);
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) s += v[k];
  int64_t tot;
  store_items(prefix, base, n, block_excl_scan(s, sh, &tot) + set.sums[blockIdx.y][blockIdx.x], v);
}

__global__ void __launch_bounds__(kScanThreads) k_scan_apply(const int32_t* __restrict__ counts,
                                                             int64_t n, const int64_t* __restrict__ sums,
                                                             int64_t* __restrict__ prefix) {
  __shared__ int64_t sh[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanItems;
  int32_t v[kScanItems];
  load_items(counts, base, n, v);
  int64_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) s += v[k];
  int64_t tot;
  store_items(prefix, base, n, block_excl_scan(s, sh, &tot) + sums[blockIdx.x], v);
}

// ---------------------------------------------------------------------------
// Leaf index: one wave per tree enumerates its leaves in ascending bit index
// (breadth-first, the order Eq. 3 counts) with ballots over 64 positions.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) k_leaf_index(const uint32_t* __restrict__ trees,
                                                    const int64_t* __restrict__ prefix,
                                                    int64_t n_trees, uint64_t* __restrict__ info) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= n_trees) return;
  const Bits b = load_bits(trees, t);
  const int64_t row0 = prefix[t];
  const uint64_t tag = (uint64_t)t << 10;
  if (!(b.lo & 1ull)) {
    if (lane_id() == 0) info[row0] = tag;
    return;
  }
  int base = 0;
  for (int c0 = 1; c0 < kNodes; c0 += 64) {
    const int i = c0 + lane_id();
    const bool leaf = i < kNodes && is_leaf(b, i);
    const uint64_t m = __ballot(leaf);
    if (leaf) info[row0 + base + __popcll(m & lanemask_lt())] = tag | (uint64_t)i;
    base += __popcll(m);
  }
}

// rowmap: one thread per voxel.
__global__ void k_rowmap(const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix,
                         int64_t n_vox, int gd, int gh, int gw, int64_t* __restrict__ rowmap) {
  const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (v >= n_vox) return;
  const int64_t W = 8LL * gw, H = 8LL * gh, D = 8LL * gd;
  int64_t r = v;
  const int vw = (int)(r % W); r /= W;
  const int vh = (int)(r % H); r /= H;
  const int vd = (int)(r % D); r /= D;
  const int64_t t = ((r * gd + (vd >> 3)) * gh + (vh >> 3)) * gw + (vw >> 3);
  const Bits b = load_bits(trees, t);
  rowmap[v] = prefix[t] + data_idx(b, leaf_at(b, vd & 7, vh & 7, vw & 7));
}

// ---------------------------------------------------------------------------
// Pool structure: thread per output tree (Eq. 10).  Input tree of octant o
// contributes its root bit as output bit 1+o and its depth-1 bits as output
// bits 9+8o+q; the output root is always split.
// ---------------------------------------------------------------------------
__global__ void k_pool_structure(const uint32_t* __restrict__ in, int64_t n_out, int gd, int gh,
                                 int gw, uint32_t* __restrict__ out, int32_t* __restrict__ counts) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_out) return;
  const int od = gd / 2, oh = gh / 2, ow = gw / 2;
  const TreePos p = tree_pos(t, od, oh, ow);
  uint64_t lo = 1ull;
  uint32_t hi = 0;
#pragma unroll
  for (int o = 0; o < 8; ++o) {
    const int a = (o >> 2) & 1, bb = (o >> 1) & 1, c = o & 1;
    const int64_t ti = ((p.n * gd + 2 * p.d + a) * gh + 2 * p.h + bb) * gw + 2 * p.w + c;
    const Bits ib = load_bits(in, ti);
    lo |= (ib.lo & 1ull) << (1 + o);
    const uint64_t d1 = (ib.lo >> 1) & 0xFFull;  // input bits 1..8
    const int pos = 9 + 8 * o;                   // output bits pos..pos+7
    if (pos + 8 <= 64) {
      lo |= d1 << pos;
    } else if (pos >= 64) {
      hi |= (uint32_t)(d1 << (pos - 64));
    } else {
      lo |= d1 << pos;
      hi |= (uint32_t)(d1 >> (64 - pos));
    }
  }
  uint4 w;
  w.x = (uint32_t)lo;
  w.y = (uint32_t)(lo >> 32);
  w.z = hi & 0x1FFu;
  w.w = 0u;
  reinterpret_cast<uint4*>(out)[t] = w;
  Bits ob;
  ob.lo = lo;
  ob.hi = w.z;
  counts[t] = n_leaves_of(ob);
}

// Unpool structure, plain (Eq. 12): thread per output tree.
__global__ void k_unpool_structure(const uint32_t* __restrict__ in, int64_t n_out, int gd, int gh,
                                   int gw, uint32_t* __restrict__ out, int32_t* __restrict__ counts) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_out) return;
  const TreePos p = tree_pos(t, 2 * gd, 2 * gh, 2 * gw);
  const int o = ((p.d & 1) << 2) | ((p.h & 1) << 1) | (p.w & 1);
  const int64_t ti = ((p.n * gd + (p.d >> 1)) * gh + (p.h >> 1)) * gw + (p.w >> 1);
  const Bits ib = load_bits(in, ti);
  uint32_t word = 0;
  if ((ib.lo & 1ull) && bit(ib, 1 + o)) {
    word = 1u;
    for (int q = 0; q < 8; ++q) word |= (uint32_t)bit(ib, 9 + 8 * o + q) << (1 + q);
  }
  uint4 w;
  w.x = word;
  w.y = w.z = w.w = 0u;
  reinterpret_cast<uint4*>(out)[t] = w;
  counts[t] = 1 + 7 * __popc(word);
}

// Guided unpool: copy the guide and check that it pools to the input.
__global__ void k_unpool_guided(const uint32_t* __restrict__ in, const uint32_t* __restrict__ guide,
                                int64_t n_in, int gd, int gh, int gw, uint32_t* __restrict__ out,
                                int32_t* __restrict__ counts, int32_t* __restrict__ mismatch) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // input tree
  if (t >= n_in) return;
  const TreePos p = tree_pos(t, gd, gh, gw);
  const int Gd = 2 * gd, Gh = 2 * gh, Gw = 2 * gw;
  uint64_t lo = 1ull;
  uint32_t hi = 0;
  for (int o = 0; o < 8; ++o) {
    const int a = (o >> 2) & 1, bb = (o >> 1) & 1, c = o & 1;
    const int64_t tg = ((p.n * Gd + 2 * p.d + a) * Gh + 2 * p.h + bb) * Gw + 2 * p.w + c;
    const uint4 gw4 = reinterpret_cast<const uint4*>(guide)[tg];
    reinterpret_cast<uint4*>(out)[tg] = gw4;
    Bits gb;
    gb.lo = (uint64_t)gw4.x | ((uint64_t)gw4.y << 32);
    gb.hi = gw4.z & 0x1FFu;
    counts[tg] = n_leaves_of(gb);
    lo |= (gb.lo & 1ull) << (1 + o);
    for (int q = 0; q < 8; ++q) {
      const int pos = 9 + 8 * o + q;
      const uint64_t v = (gb.lo >> (1 + q)) & 1ull;
      if (pos < 64) lo |= v << pos;
      else hi |= (uint32_t)v << (pos - 64);
    }
  }
  const uint4 iw = reinterpret_cast<const uint4*>(in)[t];
  const uint64_t ilo = (uint64_t)iw.x | ((uint64_t)iw.y << 32);
  if (ilo != lo || (iw.z & 0x1FFu) != hi) atomicAdd(mismatch, 1);
}

inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

}  // namespace

namespace oci {

size_t scan_workspace(int64_t n) {
  const int64_t nb = (n + kScanChunk - 1) / kScanChunk;
  return align256(sizeof(int32_t) * (size_t)n) + align256(sizeof(int64_t) * (size_t)(nb + 1)) + 256;
}

hipError_t scan_counts(const int32_t* counts, int64_t n, int64_t* prefix, void* ws,
                       hipStream_t s) {
  const int64_t nb = (n + kScanChunk - 1) / kScanChunk;
  char* p = static_cast<char*>(ws) + align256(sizeof(int32_t) * (size_t)n);
  int64_t* sums = reinterpret_cast<int64_t*>(p);
  hipLaunchKernelGGL(k_scan_reduce, dim3((unsigned)nb), dim3(kScanThreads), 0, s, counts, n, sums);
  hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(kScanThreads), 0, s, sums, nb, prefix + n);
  hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)nb), dim3(kScanThreads), 0, s, counts, n, sums, prefix);
  return hipGetLastError();
}

hipError_t scan_counts_set(int k, void* const* ws, int64_t n, int64_t* const* prefix,
                           hipStream_t s) {
  if (k < 1 || k > kMaxScans) return hipErrorInvalidValue;
  const int64_t nb = (n + kScanChunk - 1) / kScanChunk;
  ScanSet set;
  for (int i = 0; i < kMaxScans; ++i) {
    const int j = i < k ? i : 0;
    set.counts[i] = static_cast<const int32_t*>(ws[j]);
    set.prefix[i] = prefix[j];
    set.sums[i] = reinterpret_cast<int64_t*>(static_cast<char*>(ws[j]) +
                                             align256(sizeof(int32_t) * (size_t)n));
  }
  hipLaunchKernelGGL(k_scan_reduce_set, dim3((unsigned)nb, (unsigned)k), dim3(kScanThreads), 0, s,
                     set, n);
  hipLaunchKernelGGL(k_scan_sums_set, dim3(1, (unsigned)k), dim3(kScanThreads), 0, s, set, nb, n);
  hipLaunchKernelGGL(k_scan_apply_set, dim3((unsigned)nb, (unsigned)k), dim3(kScanThreads), 0, s,
                     set, n);
  return hipGetLastError();
}

int32_t* scan_counts_buffer(void* ws) { return static_cast<int32_t*>(ws); }

hipError_t launch_build(const uint8_t* occ, int n, int gd, int gh, int gw, int rule,
                        uint32_t* trees, int32_t* counts, hipStream_t s) {
  const int64_t nt = (int64_t)n * gd * gh * gw;
  const int64_t segs = (nt / gw) * ((gw + kBuildTrees - 1) / kBuildTrees);
  const int64_t blocks = (segs + kBuildSegs - 1) / kBuildSegs;
  // 16-byte loads need an even grid width (rows of 8 gw bytes on 16-byte
  // boundaries; the input itself is 16-byte aligned).
  if (gw % 2 == 0 && (reinterpret_cast<uintptr_t>(occ) & 15) == 0)
    hipLaunchKernelGGL(k_build<true>, dim3((unsigned)blocks), dim3(kBuildThreads), 0, s, occ, nt, gd, gh, gw,
                       rule, trees, counts);
  else
    hipLaunchKernelGGL(k_build<false>, dim3((unsigned)blocks), dim3(kBuildThreads), 0, s, occ, nt, gd, gh, gw,
                       rule, trees, counts);
  return hipGetLastError();
}

hipError_t launch_count(const uint32_t* trees, int64_t nt, int32_t* counts, hipStream_t s) {
  hipLaunchKernelGGL(k_count, dim3(blocks_for(nt, 256)), dim3(256), 0, s, trees, nt, counts);
  return hipGetLastError();
}

hipError_t launch_validate(const uint32_t* trees, int64_t nt, int32_t* bad, hipStream_t s) {
  hipLaunchKernelGGL(k_validate, dim3(blocks_for(nt, 256)), dim3(256), 0, s, trees, nt, bad);
  return hipGetLastError();
}

hipError_t launch_leaf_index(const uint32_t* trees, const int64_t* prefix, int64_t nt,
                             uint64_t* info, hipStream_t s) {
  hipLaunchKernelGGL(k_leaf_index, dim3(blocks_for(nt, 4)), dim3(256), 0, s, trees, prefix, nt, info);
  return hipGetLastError();
}

hipError_t launch_rowmap(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
                         int gw, int64_t* rowmap, hipStream_t s) {
  const int64_t nv = 512LL * n * gd * gh * gw;
  hipLaunchKernelGGL(k_rowmap, dim3(blocks_for(nv, 256)), dim3(256), 0, s, trees, prefix, nv, gd,
                     gh, gw, rowmap);
  return hipGetLastError();
}

hipError_t launch_pool_structure(const uint32_t* in, int n, int gd, int gh, int gw, uint32_t* out,
                                 int32_t* counts, hipStream_t s) {
  const int64_t no = (int64_t)n * (gd / 2) * (gh / 2) * (gw / 2);
  hipLaunchKernelGGL(k_pool_structure, dim3(blocks_for(no, 256)), dim3(256), 0, s, in, no, gd, gh,
                     gw, out, counts);
  return hipGetLastError();
}

hipError_t launch_unpool_structure(const uint32_t* in, const uint32_t* guide, int n, int gd, int gh,
                                   int gw, uint32_t* out, int32_t* counts, int32_t* mismatch,
                                   hipStream_t s) {
  if (guide == nullptr) {
    const int64_t no = 8LL * n * gd * gh * gw;
    hipLaunchKernelGGL(k_unpool_structure, dim3(blocks_for(no, 256)), dim3(256), 0, s, in, no, gd,
                       gh, gw, out, counts);
  } else {
    const int64_t ni = (int64_t)n * gd * gh * gw;
    hipLaunchKernelGGL(k_unpool_guided, dim3(blocks_for(ni, 256)), dim3(256), 0, s, in, guide, ni,
                       gd, gh, gw, out, counts, mismatch);
  }
  return hipGetLastError();
}

}  // namespace oci
