// Device-side helpers for the hybrid grid-octree (OctNet, Sec. 3.1).
//
// A shallow octree of depth 3 covers 8x8x8 voxels.  Its 73 split bits are
// held as two integers: lo = bits 0..63, hi = bits 64..72.  Bit indices
// 73..584 name the implicit depth-3 voxels.  The child with octant o of a
// node covers the sub-cube offset by ((o>>2)&1, (o>>1)&1, o&1) * child size
// along (d, h, w).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ocd {

constexpr int kBits = 73;    // stored split bits per tree
constexpr int kNodes = 585;  // 1 + 8 + 64 + 512

struct Bits {
  uint64_t lo;  // bits 0..63
  uint32_t hi;  // bits 64..72 (positions 0..8)
};

__device__ __forceinline__ Bits load_bits(const uint32_t* __restrict__ trees, int64_t t) {
  const uint4 w = reinterpret_cast<const uint4*>(trees)[t];
  Bits b;
  b.lo = (uint64_t)w.x | ((uint64_t)w.y << 32);
  b.hi = w.z & 0x1FFu;
  return b;
}

__host__ __device__ __forceinline__ int bit(const Bits& b, int i) {
  if (i < 64) return (int)((b.lo >> i) & 1ull);
  if (i < kBits) return (int)((b.hi >> (i - 64)) & 1u);
  return 0;
}

// Number of set bits among bit indices [0, n).
__device__ __forceinline__ int popc_below(const Bits& b, int n) {
  if (n <= 0) return 0;
  if (n < 64) return __popcll(b.lo & ((1ull << n) - 1ull));
  int m = n - 64;
  if (m > 9) m = 9;
  return __popcll(b.lo) + __popc(b.hi & ((1u << m) - 1u));
}

__device__ __forceinline__ int popc_all(const Bits& b) { return __popcll(b.lo) + __popc(b.hi); }

// Eq. 3: offset of leaf i inside its tree's data block (breadth-first order).
// For i = 0 (an unsplit root, the only leaf) the offset is 0.
__device__ __forceinline__ int data_idx(const Bits& b, int i) {
  if (i == 0) return 0;
  const int pa = (i - 1) >> 3;  // Eq. 1
  return 8 * popc_below(b, pa) + 1 - popc_below(b, i) + ((i - 1) & 7);
}

__device__ __forceinline__ int n_leaves_of(const Bits& b) { return 1 + 7 * popc_all(b); }

// Bit index of the leaf that holds local voxel (d, h, w), each in [0, 8).
__device__ __forceinline__ int leaf_at(const Bits& b, int d, int h, int w) {
  if (!(b.lo & 1ull)) return 0;
  const int o1 = (((d >> 2) & 1) << 2) | (((h >> 2) & 1) << 1) | ((w >> 2) & 1);
  const int n1 = 1 + o1;
  if (!bit(b, n1)) return n1;
  const int o2 = (((d >> 1) & 1) << 2) | (((h >> 1) & 1) << 1) | ((w >> 1) & 1);
  const int n2 = 8 * n1 + 1 + o2;  // Eq. 2
  if (!bit(b, n2)) return n2;
  const int o3 = ((d & 1) << 2) | ((h & 1) << 1) | (w & 1);
  return 8 * n2 + 1 + o3;
}

// Depth, local origin and size of node i.
struct Cell {
  int depth, d, h, w, size;
};

__host__ __device__ __forceinline__ Cell cell_of(int i) {
  Cell c;
  if (i == 0) {
    c.depth = 0; c.d = c.h = c.w = 0; c.size = 8;
    return c;
  }
  int o1, o2 = -1, o3 = -1;
  if (i < 9) {
    o1 = i - 1;
    c.depth = 1; c.size = 4;
  } else if (i < 73) {
    const int q = i - 9;
    o1 = q >> 3; o2 = q & 7;
    c.depth = 2; c.size = 2;
  } else {
    const int q = i - 73;
    o1 = q >> 6; o2 = (q >> 3) & 7; o3 = q & 7;
    c.depth = 3; c.size = 1;
  }
  c.d = 4 * ((o1 >> 2) & 1); c.h = 4 * ((o1 >> 1) & 1); c.w = 4 * (o1 & 1);
  if (o2 >= 0) { c.d += 2 * ((o2 >> 2) & 1); c.h += 2 * ((o2 >> 1) & 1); c.w += 2 * (o2 & 1); }
  if (o3 >= 0) { c.d += (o3 >> 2) & 1; c.h += (o3 >> 1) & 1; c.w += o3 & 1; }
  return c;
}

// Is node i a leaf of the tree (exists and not split)?
__device__ __forceinline__ bool is_leaf(const Bits& b, int i) {
  if (i == 0) return !(b.lo & 1ull);
  const int p = (i - 1) >> 3;
  return bit(b, p) && (i >= kBits || !bit(b, i));
}

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Tree linear index -> (sample, td, th, tw).
struct TreePos {
  int64_t n;
  int d, h, w;
};

__device__ __forceinline__ TreePos tree_pos(int64_t t, int gd, int gh, int gw) {
  TreePos p;
  if ((uint64_t)t < (1ull << 32)) {
    // 32-bit divisions (every grid here has fewer than 2^32 trees; the
    // 64-bit ones cost several times more).
    uint32_t u = (uint32_t)t;
    p.w = (int)(u % (uint32_t)gw); u /= (uint32_t)gw;
    p.h = (int)(u % (uint32_t)gh); u /= (uint32_t)gh;
    p.d = (int)(u % (uint32_t)gd); u /= (uint32_t)gd;
    p.n = (int64_t)u;
    return p;
  }
  p.w = (int)(t % gw); t /= gw;
  p.h = (int)(t % gh); t /= gh;
  p.d = (int)(t % gd); t /= gd;
  p.n = t;
  return p;
}

}  // namespace ocd
