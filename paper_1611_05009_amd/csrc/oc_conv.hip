// Grid-octree 3x3x3 convolution (OctNet Eq. 8 with average pooling).
//
// For a leaf with cell Omega (origin o, edge s) the output is
//   out[co] = b[co] + (1/s^3) * sum_{delta in {-1,0,1}^3} sum_ci
//             W[co][ci][1-delta] * S_delta[ci],
//   S_delta[ci] = sum of the input over the shifted cell Omega + delta
// (Eq. 7 pairs input offset delta with tap 1 - delta).  S_delta is a sum over
// the leaves that intersect the cell grown by one voxel, each weighted by the
// per-axis overlap of its cell with the shifted window; the cell's own value
// covers the part of the window inside the cell.  This is the paper's
// observation that the response inside a cell is constant up to its boundary
// (Sec. 3.2 and the supplement's "Efficient Convolution"), turned into 27
// window sums followed by one (27*Cin) x Cout contraction per leaf.
#include <mutex>
#include <type_traits>

#include "oc_internal.h"

// Tuning knobs (compile-time): deltas of gathered A rows in flight in the
// unit-voxel kernel; shell voxels / regions per scheduling group in the cell
// kernels.
#ifndef OC_UNIT_ACCS
#define OC_UNIT_ACCS 1
#endif
#ifndef OC_UNIT_PREFETCH
#define OC_UNIT_PREFETCH 2
#endif
// Deltas of gathers in flight where a lane's row piece is small (at most
// OC_UNIT_SMALL_CH floats per lane per delta, so more deltas fit in
// registers): the narrow layers are bound by the gathers, not by the
// matrix unit.
#ifndef OC_UNIT_PREFETCH_SMALL
#define OC_UNIT_PREFETCH_SMALL 8
#endif
#ifndef OC_UNIT_SMALL_CH
#define OC_UNIT_SMALL_CH 2
#endif
template <int CIN, int MS>
constexpr int unit_prefetch() {
  return CIN / (MS == 32 ? 2 : 4) <= OC_UNIT_SMALL_CH ? OC_UNIT_PREFETCH_SMALL : OC_UNIT_PREFETCH;
}
using namespace ocd;

namespace {

constexpr int kThreads = 256;

// ---------------------------------------------------------------------------
// Weights: wt[(didx*cin + ci)*cout + co] = w[co][ci][1-dd][1-dh][1-dw]
// with didx = (dd+1)*9 + (dh+1)*3 + (dw+1).
// ---------------------------------------------------------------------------
__global__ void k_transpose_weights(const float* __restrict__ w, int cin, int cout,
                                    float* __restrict__ wt) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = 27LL * cin * cout;
  if (idx >= total) return;
  const int co = (int)(idx % cout);
  const int64_t k = idx / cout;
  const int ci = (int)(k % cin);
  const int didx = (int)(k / cin);
  const int dd = didx / 9 - 1, dh = (didx / 3) % 3 - 1, dw = didx % 3 - 1;
  const int tap = (1 - dd) * 9 + (1 - dh) * 3 + (1 - dw);
  wt[idx] = w[((int64_t)co * cin + ci) * 27 + tap];
}

// ---------------------------------------------------------------------------
// Shell enumeration.
// Region r (r = didx, r != 13) of a leaf is the part of the one-voxel shell
// around the cell in direction (dd, dh, dw): per axis [o-1, o) for -1,
// [o, o+s) for 0 and [o+s, o+s+1) for +1.  A region lies inside one tree.
// Every leaf that intersects a region gives one entry: its row and, per
// axis, the intersection interval relative to o-1 (4 bits per end).
// ---------------------------------------------------------------------------
struct Entry {
  uint32_t row;
  uint32_t iv;  // axis a: bits [8a, 8a+4) = start, [8a+4, 8a+8) = end, relative to o-1
};

// Slot capacity of region r for the largest cell (s = 8): the number of unit
// voxels in the region.  Offsets are the running sums; the self entry uses
// slot kSelfSlot.
struct SlotTable {
  int off[27];
};
constexpr SlotTable make_slot_table() {
  SlotTable t{};
  int acc = 0;
  for (int r = 0; r < 27; ++r) {
    t.off[r] = acc;
    if (r == 13) continue;
    const int dd = r / 9 - 1, dh = (r / 3) % 3 - 1, dw = r % 3 - 1;
    acc += (dd == 0 ? 8 : 1) * (dh == 0 ? 8 : 1) * (dw == 0 ? 8 : 1);
  }
  return t;
}
__constant__ SlotTable c_slots = make_slot_table();

// Edge-2 cells.  The shell is the 56 voxels u of the 4^3 block [o-1, o+3)
// outside [o, o+2) (u in [0,4)^3 minus [1,2]^3); voxel u lies in the window
// of delta iff u_a - delta_a - 1 is in {0, 1} on every axis.
constexpr int shell2_u(int q) {
  int k = 0;
  for (int u = 0; u < 64; ++u) {
    const int ud = u >> 4, uh = (u >> 2) & 3, uw = u & 3;
    const bool inner = ud >= 1 && ud <= 2 && uh >= 1 && uh <= 2 && uw >= 1 && uw <= 2;
    if (inner) continue;
    if (k == q) return u;
    ++k;
  }
  return -1;
}

// Index in that list of shell voxel u (-1 for the cell's own voxels).
constexpr int shell2_q(int u) {
  for (int q = 0; q < 56; ++q)
    if (shell2_u(q) == u) return q;
  return -1;
}

struct Shell2Table {
  uint8_t u[56];
};
constexpr Shell2Table make_shell2_table() {
  Shell2Table t{};
  for (int q = 0; q < 56; ++q) t.u[q] = (uint8_t)shell2_u(q);
  return t;
}
__constant__ Shell2Table c_shell2 = make_shell2_table();
constexpr int kSlots = 6 * 64 + 12 * 8 + 8 + 1;  // 489
constexpr int kSelfSlot = kSlots - 1;
// Entries of a split depth-1 node's table: the 6^3 voxels around its 4^3.
constexpr int kNodeEntries = 216;

__device__ __forceinline__ uint32_t pack_iv(int a0, int a1, int b0, int b1, int c0, int c1) {
  return (uint32_t)(a0 | (a1 << 4) | (b0 << 8) | (b1 << 12) | (c0 << 16) | (c1 << 20));
}

// Overlap of relative interval [lo, hi) with the window of shift delta,
// [delta+1, delta+1+s).
__device__ __forceinline__ float ov(int lo, int hi, int delta, int s) {
  const int a = max(lo, delta + 1), b = min(hi, delta + 1 + s);
  return (float)max(0, b - a);
}

struct LeafGeo {
  int64_t n;         // sample
  int od, oh, ow;    // global voxel origin
  int s;             // edge length
  int64_t row;
};

__device__ __forceinline__ LeafGeo leaf_geo(uint64_t info, int64_t row, int gd, int gh, int gw) {
  LeafGeo g;
  const int64_t t = (int64_t)(info >> 10);
  const int bit_i = (int)(info & 1023u);
  const TreePos p = tree_pos(t, gd, gh, gw);
  const Cell c = cell_of(bit_i);
  g.n = p.n;
  g.od = 8 * p.d + c.d;
  g.oh = 8 * p.h + c.h;
  g.ow = 8 * p.w + c.w;
  g.s = c.size;
  g.row = row;
  return g;
}

// Enumerate the leaves of region r of leaf g into slots [off, off+cap);
// returns the number of entries.
__device__ int enumerate_region(const LeafGeo& g, int r, const uint32_t* __restrict__ trees,
                                const int64_t* __restrict__ prefix, int gd, int gh, int gw,
                                Entry* __restrict__ slots) {
  const int dir[3] = {r / 9 - 1, (r / 3) % 3 - 1, r % 3 - 1};
  const int org[3] = {g.od, g.oh, g.ow};
  const int lim[3] = {8 * gd, 8 * gh, 8 * gw};
  int lo[3], hi[3];
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    if (dir[a] < 0) { lo[a] = org[a] - 1; hi[a] = org[a]; }
    else if (dir[a] == 0) { lo[a] = org[a]; hi[a] = org[a] + g.s; }
    else { lo[a] = org[a] + g.s; hi[a] = org[a] + g.s + 1; }
    if (lo[a] < 0 || hi[a] > lim[a]) return 0;  // outside the grid: zero padding
  }
  const int T[3] = {lo[0] >> 3, lo[1] >> 3, lo[2] >> 3};
  const int64_t t = ((g.n * gd + T[0]) * gh + T[1]) * gw + T[2];
  const Bits b = load_bits(trees, t);
  const int64_t row0 = prefix[t];
  int L[3], Hh[3], base[3];
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    base[a] = 8 * T[a];
    L[a] = lo[a] - base[a];
    Hh[a] = hi[a] - base[a];
  }
  int cnt = 0;
  // emit a leaf with local cell (cd, ch, cw, size)
  auto emit = [&](int node, int cd, int ch, int cw, int size) {
    const int c[3] = {cd, ch, cw};
    int iv[6];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      const int x0 = max(c[a], L[a]) + base[a] - (org[a] - 1);
      const int x1 = min(c[a] + size, Hh[a]) + base[a] - (org[a] - 1);
      iv[2 * a] = x0;
      iv[2 * a + 1] = x1;
    }
    Entry e;
    e.row = (uint32_t)(row0 + data_idx(b, node));
    e.iv = pack_iv(iv[0], iv[1], iv[2], iv[3], iv[4], iv[5]);
    slots[cnt++] = e;
  };
  auto hit = [&](int cd, int ch, int cw, int size) {
    return L[0] < cd + size && cd < Hh[0] && L[1] < ch + size && ch < Hh[1] && L[2] < cw + size &&
           cw < Hh[2];
  };
  if (!(b.lo & 1ull)) {
    emit(0, 0, 0, 0, 8);
    return cnt;
  }
  for (int o1 = 0; o1 < 8; ++o1) {
    const int d1 = 4 * ((o1 >> 2) & 1), h1 = 4 * ((o1 >> 1) & 1), w1 = 4 * (o1 & 1);
    if (!hit(d1, h1, w1, 4)) continue;
    const int n1 = 1 + o1;
    if (!bit(b, n1)) { emit(n1, d1, h1, w1, 4); continue; }
    for (int o2 = 0; o2 < 8; ++o2) {
      const int d2 = d1 + 2 * ((o2 >> 2) & 1), h2 = h1 + 2 * ((o2 >> 1) & 1), w2 = w1 + 2 * (o2 & 1);
      if (!hit(d2, h2, w2, 2)) continue;
      const int n2 = 8 * n1 + 1 + o2;
      if (!bit(b, n2)) { emit(n2, d2, h2, w2, 2); continue; }
      for (int o3 = 0; o3 < 8; ++o3) {
        const int d3 = d2 + ((o3 >> 2) & 1), h3 = h2 + ((o3 >> 1) & 1), w3 = w2 + (o3 & 1);
        if (!hit(d3, h3, w3, 1)) continue;
        emit(8 * n2 + 1 + o3, d3, h3, w3, 1);
      }
    }
  }
  return cnt;
}

// Window sums of one leaf into s_out[27][cin] (LDS).  Called by a whole wave:
// lanes 0..25 enumerate the 26 shell regions, then lanes run over channels.
__device__ void window_sums(const LeafGeo& g, const uint32_t* __restrict__ trees,
                            const int64_t* __restrict__ prefix, int gd, int gh, int gw,
                            const float* __restrict__ in, int cin, Entry* __restrict__ slots,
                            int* __restrict__ counts, float* __restrict__ s_out) {
  const int lane = lane_id();
  if (lane < 27) {
    const int r = lane;
    int cnt;
    if (r == 13) {
      Entry e;
      e.row = (uint32_t)g.row;
      e.iv = pack_iv(1, g.s + 1, 1, g.s + 1, 1, g.s + 1);
      slots[kSelfSlot] = e;
      cnt = 1;
    } else {
      cnt = enumerate_region(g, r, trees, prefix, gd, gh, gw, slots + c_slots.off[r]);
    }
    counts[r] = cnt;
  }
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
  for (int c0 = 0; c0 < cin; c0 += 64) {
    const int ci = c0 + lane;
    float S[27];
#pragma unroll
    for (int k = 0; k < 27; ++k) S[k] = 0.f;
    for (int r = 0; r < 27; ++r) {
      const int cnt = counts[r];
      const Entry* es = slots + (r == 13 ? kSelfSlot : c_slots.off[r]);
      for (int e = 0; e < cnt; ++e) {
        const Entry en = es[e];
        const float x = ci < cin ? in[(int64_t)en.row * cin + ci] : 0.f;
        const int iv = (int)en.iv;
        float cd[3], ch[3], cw[3];
#pragma unroll
        for (int dl = 0; dl < 3; ++dl) {
          cd[dl] = ov(iv & 15, (iv >> 4) & 15, dl - 1, g.s);
          ch[dl] = ov((iv >> 8) & 15, (iv >> 12) & 15, dl - 1, g.s);
          cw[dl] = ov((iv >> 16) & 15, (iv >> 20) & 15, dl - 1, g.s);
        }
#pragma unroll
        for (int a = 0; a < 3; ++a)
#pragma unroll
          for (int bb = 0; bb < 3; ++bb) {
            const float xab = x * cd[a] * ch[bb];
#pragma unroll
            for (int c = 0; c < 3; ++c) S[a * 9 + bb * 3 + c] += xab * cw[c];
          }
      }
    }
    if (ci < cin) {
#pragma unroll
      for (int k = 0; k < 27; ++k) s_out[k * cin + ci] = S[k];
    }
  }
}

// ---------------------------------------------------------------------------
// Generic kernel: tiles of `tm` rows, taken from `rows_list` (its length in
// *n_list) or, without a list, rows 0..n_leaves-1.  Waves compute window sums
// into LDS, then all threads run the VALU contraction.  Grid-stride over
// tiles, so the grid does not depend on the list length.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kThreads) k_conv_generic(
    const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix,
    const uint64_t* __restrict__ info, int64_t n_leaves, int gd, int gh, int gw,
    const float* __restrict__ in, int cin, const float* __restrict__ wt,
    const float* __restrict__ bias, int cout, int relu, float* __restrict__ out, int tm,
    const int32_t* __restrict__ rows_list, const int64_t* __restrict__ n_list) {
  extern __shared__ float smem[];
  // layout: [4 waves][kSlots] entries, [4][32] counts, [tm] rows, [tm][27*cin] sums, [tm] scale
  Entry* slots_all = reinterpret_cast<Entry*>(smem);
  int* counts_all = reinterpret_cast<int*>(slots_all + 4 * kSlots);
  int64_t* rowv = reinterpret_cast<int64_t*>(counts_all + 4 * 32);
  float* sums = reinterpret_cast<float*>(rowv + 32);
  float* scale = sums + (int64_t)tm * 27 * cin;
  const int wv = threadIdx.x >> 6;
  const int64_t n_rows = rows_list ? *n_list : n_leaves;
  const int64_t n_tiles = (n_rows + tm - 1) / tm;
  const int K = 27 * cin;
  for (int64_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    const int64_t base = tile * tm;
    for (int m = wv; m < tm; m += 4) {
      const int64_t idx = base + m;
      if (idx < n_rows) {
        const int64_t row = rows_list ? (int64_t)rows_list[idx] : idx;
        if (row < 0 || row >= n_leaves) {  // only a non-canonical structure gets here
          if (lane_id() == 0) rowv[m] = -1;
          __builtin_amdgcn_wave_barrier();
          continue;
        }
        const LeafGeo g = leaf_geo(info[row], row, gd, gh, gw);
        window_sums(g, trees, prefix, gd, gh, gw, in, cin, slots_all + wv * kSlots,
                    counts_all + wv * 32, sums + (int64_t)m * K);
        if (lane_id() == 0) {
          scale[m] = 1.f / (float)(g.s * g.s * g.s);
          rowv[m] = row;
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < tm * cout; idx += kThreads) {
      const int m = idx / cout, co = idx % cout;
      if (base + m >= n_rows || rowv[m] < 0) continue;
      const float* sm = sums + (int64_t)m * K;
      float acc = 0.f;
      for (int k = 0; k < K; ++k) acc = fmaf(sm[k], wt[(int64_t)k * cout + co], acc);
      float v = acc * scale[m] + (bias ? bias[co] : 0.f);
      if (relu) v = fmaxf(v, 0.f);
      out[rowv[m] * cout + co] = v;
    }
    __syncthreads();  // the next tile reuses the LDS
  }
}

// LDS budget: 16 KB of shell entries plus at most 44 KB of window sums, so a
// block stays within 64 KB for every cin <= 256.
int generic_tile(int cin) {
  int tm = 45056 / (108 * cin);
  if (tm > 32) tm = 32;
  if (tm < 1) tm = 1;
  return tm;
}

size_t generic_smem(int cin, int tm) {
  return sizeof(Entry) * 4 * kSlots + sizeof(int) * 4 * 32 + sizeof(int64_t) * 32 +
         sizeof(float) * (size_t)tm * 27 * cin + sizeof(float) * tm;
}

// ---------------------------------------------------------------------------
// Unit-voxel groups.
// In breadth-first order the leaves of a tree with bit index < 73 (cells of
// edge 2, 4, 8) come first, then the depth-3 voxels, eight consecutive rows
// per split depth-2 node in ascending node order.  A group is one split
// depth-2 node: key = tree << 6 | (node - 9); its rows are
// prefix[tree] + n_big(tree) + 8k .. +8 for the k-th split depth-2 node.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int depth2_splits(const Bits& b) {
  return __popcll(b.lo >> 9) + __popc(b.hi);
}

// Kinds of larger cells, in the order the lists hold them: edge-8 cells
// whose 18 face and edge neighbours (inside the grid) are unsplit trees, the
// other edge-8 cells, edge-4 cells, edge-2 cells.
constexpr int kKinds = 4;

// Per-tree counts: unit-voxel groups (split depth-2 nodes), each kind of
// larger cell, boundary-sum slots and split depth-1 nodes (node tables).  Edge-8 cells are unsplit trees,
// edge-4 cells unsplit depth-1 nodes of a split root, edge-2 cells unsplit
// depth-2 nodes of a split depth-1 node.  A split tree has one slot for
// itself and one per split depth-1 node.
__global__ void k_leaf_kinds(const uint32_t* __restrict__ trees, int64_t n_trees, int gd, int gh,
                             int gw, int32_t* __restrict__ n_grp, int32_t* __restrict__ n8t,
                             int32_t* __restrict__ n8n, int32_t* __restrict__ n4,
                             int32_t* __restrict__ n2, int32_t* __restrict__ nslot,
                             int32_t* __restrict__ nd1) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_trees) return;
  const Bits b = load_bits(trees, t);
  const int root = (int)(b.lo & 1ull);
  const int p1 = __popc((uint32_t)(b.lo >> 1) & 0xFFu);
  const int p2 = depth2_splits(b);
  int trivial = 0;
  if (!root) {
    // Trivial: no face or edge neighbour tree is split.  All 18 root bits
    // are read at once (a neighbour outside the grid reads the tree's own,
    // unsplit, root bit).
    const TreePos p = tree_pos(t, gd, gh, gw);
    uint32_t split = 0u;
#pragma unroll
    for (int r = 0; r < 27; ++r) {
      const int dd = r / 9 - 1, dh = (r / 3) % 3 - 1, dw = r % 3 - 1;
      const int nz = (dd != 0) + (dh != 0) + (dw != 0);
      if (nz != 1 && nz != 2) continue;
      const int qd = p.d + dd, qh = p.h + dh, qw = p.w + dw;
      const bool in = qd >= 0 && qh >= 0 && qw >= 0 && qd < gd && qh < gh && qw < gw;
      const int64_t q = in ? ((p.n * gd + qd) * gh + qh) * gw + qw : t;
      split |= trees[4 * q];
    }
    trivial = (split & 1u) ? 0 : 1;
  }
  n_grp[t] = p2;
  n8t[t] = (!root && trivial) ? 1 : 0;
  n8n[t] = (!root && !trivial) ? 1 : 0;
  n4[t] = root ? 8 - p1 : 0;
  n2[t] = max(0, 8 * p1 - p2);
  nslot[t] = root ? 1 + p1 : 0;
  nd1[t] = root ? p1 : 0;
}

// Leaf lists.  gkey: one key per unit-voxel group.  brow: the rows of every
// larger cell, grouped by kind (tree order within a kind), so that a tile of
// consecutive entries of one kind holds cells of one size.  stl: the split
// trees in order (there are n_trees - meta[0] - meta[1]).
// meta = {count of each kind, total}.
__global__ void k_leaf_lists(const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix,
                             const int64_t* __restrict__ gpre, const int64_t* __restrict__ p8t,
                             const int64_t* __restrict__ p8n, const int64_t* __restrict__ p4,
                             const int64_t* __restrict__ p2, const int64_t* __restrict__ d1pre,
                             int64_t n_trees, int64_t* __restrict__ gkey, int32_t* __restrict__ brow,
                             int64_t gcap, int64_t bcap, int32_t* __restrict__ stl,
                             int64_t* __restrict__ meta, int32_t* __restrict__ e2key, int64_t e2cap,
                             int64_t* __restrict__ bkey, int64_t kcap) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n_trees) return;
  const int64_t c8t = p8t[n_trees], c8n = p8n[n_trees], c4 = p4[n_trees], c2 = p2[n_trees];
  if (t == 0) {
    meta[0] = c8t;
    meta[1] = c8n;
    meta[2] = c4;
    meta[3] = c2;
    meta[4] = c8t + c8n + c4 + c2;
  }
  const Bits b = load_bits(trees, t);
  const int64_t row0 = prefix[t];
  // The capacities only matter for a non-canonical structure, whose counts
  // need not match the leaf total the buffers were sized for.
  auto put = [&](int64_t k, int64_t row) {
    if (k >= 0 && k < bcap) brow[k] = (int32_t)row;
  };
  // bkey: tree << 10 | bit index of the edge-8 and edge-4 cells' entries.
  auto key = [&](int64_t k, int bi) {
    if (k >= 0 && k < kcap) bkey[k] = (t << 10) | bi;
  };
  if (p8t[t + 1] > p8t[t]) {
    put(p8t[t], row0);
    key(p8t[t], 0);
  }
  if (p8n[t + 1] > p8n[t]) {
    put(c8t + p8n[t], row0);
    key(c8t + p8n[t], 0);
  }
  if (b.lo & 1ull) stl[t - p8t[t] - p8n[t]] = (int32_t)t;
  const int64_t n4t = p4[t + 1] - p4[t];
  for (int64_t k = p4[t]; k < p4[t + 1]; ++k) put(c8t + c8n + k, row0 + (k - p4[t]));
  if (b.lo & 1ull) {
    int64_t k = c8t + c8n + p4[t];
    for (int o1 = 0; o1 < 8; ++o1)
      if (!bit(b, 1 + o1)) key(k++, 1 + o1);
  }
  for (int64_t k = p2[t]; k < p2[t + 1]; ++k) put(c8t + c8n + c4 + k, row0 + n4t + (k - p2[t]));
  // Edge-2 cells in the same order (ascending bit index): the split
  // depth-1 node holding each (its index in the node tables) and its octant.
  if (b.lo & 1ull) {
    int64_t k2 = p2[t], node = d1pre[t];
    for (int o1 = 0; o1 < 8; ++o1) {
      if (!bit(b, 1 + o1)) continue;
      for (int o2 = 0; o2 < 8; ++o2) {
        if (bit(b, 9 + 8 * o1 + o2)) continue;
        if (k2 >= 0 && k2 < e2cap && node < (1LL << 28)) e2key[k2] = (int32_t)((node << 3) | o2);
        ++k2;
      }
      ++node;
    }
  }
  int64_t k = gpre[t];
  uint64_t m = b.lo >> 9;  // bits 9..63 -> positions 0..54
  while (m && k < gcap) {
    const int q = __ffsll((unsigned long long)m) - 1;
    m &= m - 1;
    gkey[k++] = (t << 6) | q;
  }
  uint32_t h = b.hi;  // bits 64..72 -> q = 55..63
  while (h && k < gcap) {
    const int q = __ffs(h) - 1;
    h &= h - 1;
    gkey[k++] = (t << 6) | (55 + q);
  }
}


// Voxel u of the 4^3 neighbourhood of group `key`, split into its tree (-1
// outside the grid) and its local position (d<<6 | h<<3 | w): the address
// part of neighbour_row, so that the tree loads can be issued early.
struct NbProbe {
  int64_t tt;
  int local;
};

__device__ __forceinline__ NbProbe neighbour_probe(int gd, int gh, int gw, int64_t key, int u) {
  NbProbe r;
  r.tt = -1;
  r.local = 0;
  if (key < 0) return r;
  const int64_t t = key >> 6;
  const int q = (int)(key & 63);
  const TreePos p = tree_pos(t, gd, gh, gw);
  const int o1 = q >> 3, o2 = q & 7;
  const int vd = 8 * p.d + 4 * ((o1 >> 2) & 1) + 2 * ((o2 >> 2) & 1) - 1 + (u >> 4);
  const int vh = 8 * p.h + 4 * ((o1 >> 1) & 1) + 2 * ((o2 >> 1) & 1) - 1 + ((u >> 2) & 3);
  const int vw = 8 * p.w + 4 * (o1 & 1) + 2 * (o2 & 1) - 1 + (u & 3);
  if (vd < 0 || vh < 0 || vw < 0 || vd >= 8 * gd || vh >= 8 * gh || vw >= 8 * gw) return r;
  r.tt = ((p.n * gd + (vd >> 3)) * gh + (vh >> 3)) * gw + (vw >> 3);
  r.local = ((vd & 7) << 6) | ((vh & 7) << 3) | (vw & 7);
  return r;
}

// Row of the leaf holding voxel u (u = 16 ud + 4 uh + uw, each in 0..3) of
// the 4^3 neighbourhood [p-1, p+3) of the group's 2^3 block at origin p;
// -1 outside the grid (zero padding).
__device__ __forceinline__ int32_t neighbour_row(const uint32_t* __restrict__ trees,
                                                 const int64_t* __restrict__ prefix, int gd, int gh,
                                                 int gw, int64_t key, int u) {
  const int64_t t = key >> 6;
  const int q = (int)(key & 63);
  const TreePos p = tree_pos(t, gd, gh, gw);
  const int o1 = q >> 3, o2 = q & 7;
  const int vd = 8 * p.d + 4 * ((o1 >> 2) & 1) + 2 * ((o2 >> 2) & 1) - 1 + (u >> 4);
  const int vh = 8 * p.h + 4 * ((o1 >> 1) & 1) + 2 * ((o2 >> 1) & 1) - 1 + ((u >> 2) & 3);
  const int vw = 8 * p.w + 4 * (o1 & 1) + 2 * (o2 & 1) - 1 + (u & 3);
  if (vd < 0 || vh < 0 || vw < 0 || vd >= 8 * gd || vh >= 8 * gh || vw >= 8 * gw) return -1;
  const int64_t tt = ((p.n * gd + (vd >> 3)) * gh + (vh >> 3)) * gw + (vw >> 3);
  const Bits b = load_bits(trees, tt);
  return (int32_t)(prefix[tt] + data_idx(b, leaf_at(b, vd & 7, vh & 7, vw & 7)));
}

// ---------------------------------------------------------------------------
// MFMA kernel for unit voxels.
//
// A wave owns a tile of MS rows = MS/8 groups.  For a unit voxel the window
// sum S_delta is the input row of the leaf holding voxel o + delta, so the
// contraction out = sum_delta W[1-delta] x(o+delta) is an implicit GEMM
// (M = rows, K = 27 cin, N = cout) whose A rows are gathered from the input.
//   MS = 32: v_mfma_f32_32x32x2_f32, lane l: A row l%32, k-slot l/32,
//            B column l%32; D[8(r/4) + 4(l/32) + r%4][l%32] in register r.
//   MS = 16: v_mfma_f32_16x16x4_f32, lane l: A row l%16, k-slot l/16,
//            B column l%16; D[4(l/16) + r][l%16] in register r.
// The K index (delta, ci) is ordered so that a lane of k-slot g holds CH
// channels of its row in NV vectors of VEC: vector v holds channels
// VEC (KS v + g) .. + VEC - 1 (KS = k-slots).  One load instruction then
// reads, per row, KS * VEC consecutive channels, whole 64-byte sectors where
// the row allows, instead of touching every sector of the row each time.
// Weights live in LDS already in B-operand order; NT N-tiles of MS columns
// cover cout (padded with zero weights).
// ---------------------------------------------------------------------------
template <int CIN, int NT, int MS>
struct MfmaCfg {
  static constexpr int KS = MS == 32 ? 2 : 4;  // k-slots per MFMA
  static constexpr int CH = CIN / KS;          // channels per lane per delta
  static constexpr int VEC = CH % 4 == 0 ? 4 : (CH % 2 == 0 ? 2 : 1);
  static constexpr int NV = CH / VEC;
  static constexpr int VSTRIDE = KS * VEC;     // channels between a lane's vectors
  static constexpr int GROUPS = MS / 8;
  static constexpr int NCOL = MS * NT;
  static constexpr int WFLOATS = 27 * CIN * NCOL;
  static_assert(CIN % KS == 0, "cin must split over the k-slots");
};

template <int V> struct VecT;
template <> struct VecT<1> { typedef float type; };
template <> struct VecT<2> { typedef float __attribute__((ext_vector_type(2))) type; };
template <> struct VecT<4> { typedef float __attribute__((ext_vector_type(4))) type; };

template <int MS> struct AccT;
template <> struct AccT<32> { typedef float __attribute__((ext_vector_type(16))) type; };
template <> struct AccT<16> { typedef float __attribute__((ext_vector_type(4))) type; };

template <int MS>
__device__ __forceinline__ typename AccT<MS>::type mfma(float a, float b, typename AccT<MS>::type c);
template <>
__device__ __forceinline__ AccT<32>::type mfma<32>(float a, float b, AccT<32>::type c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}
template <>
__device__ __forceinline__ AccT<16>::type mfma<16>(float a, float b, AccT<16>::type c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

template <int V>
__device__ __forceinline__ float vget(const typename VecT<V>::type& v, int i) {
  if constexpr (V == 1) return v;
  else return v[i];
}

// Tile schedule of a wave.  Workgroups are dispatched round-robin over the 8
// XCDs, each with its own L2.  XCD x owns the x-th eighth of the tiles (a
// compact region of space), and its waves interleave over that region, so
// the tiles in flight on one XCD at any time are neighbours that share
// gathered input rows in L2.  Tiles: first, first + stride, ... < end.
struct WaveTiles {
  int64_t first, end, stride;
};

__device__ __forceinline__ WaveTiles wave_tiles(int64_t n_tiles) {
  const int nwaves = blockDim.x >> 6, wave = threadIdx.x >> 6;
  const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8, xblocks = gridDim.x / 8;
  const int64_t per = (n_tiles + 7) / 8;
  WaveTiles t;
  t.end = min(n_tiles, (int64_t)(xcd + 1) * per);
  t.first = (int64_t)xcd * per + (int64_t)slot * nwaves + wave;
  t.stride = (int64_t)xblocks * nwaves;
  return t;
}

// The same schedule for workgroups whose waves all work on one tile.
__device__ __forceinline__ WaveTiles group_tiles(int64_t n_tiles) {
  const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8, xblocks = gridDim.x / 8;
  const int64_t per = (n_tiles + 7) / 8;
  WaveTiles t;
  t.end = min(n_tiles, (int64_t)(xcd + 1) * per);
  t.first = (int64_t)xcd * per + slot;
  t.stride = xblocks;
  return t;
}

// Gathers of input rows use raw buffer loads: one resource covers the input
// (in_bytes valid bytes), offsets are 32-bit, and an offset past the end
// reads as zero, which is the zero padding outside the grid.
constexpr uint32_t kOutside = 0xFFFF0000u;  // offset of a voxel outside the grid

__device__ __forceinline__ __amdgpu_buffer_rsrc_t input_rsrc(const float* in, uint32_t in_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(in), (short)0, (int)in_bytes,
                                           0x00020000);
}

template <int V>
__device__ __forceinline__ typename VecT<V>::type gather(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  if constexpr (V == 4)
    return __builtin_bit_cast(typename VecT<4>::type, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
  else if constexpr (V == 2)
    return __builtin_bit_cast(typename VecT<2>::type, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
  else
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

// Byte offset of channel ch of a row (kOutside for row < 0).
template <int CIN>
__device__ __forceinline__ uint32_t row_offset(int row, int ch) {
  return row < 0 ? kOutside : (uint32_t)row * (uint32_t)(CIN * 4) + (uint32_t)(ch * 4);
}

// The forward kernels gather rows by row index through one of two policies
// (the host picks one per launch):
//   RowsRaw:  one raw buffer resource over the input, 32-bit byte offsets
//             row * 4 CIN + off; the row index kNoRow wraps to an offset
//             past the end, which reads zero (the padding outside the grid).
//             For inputs below 4 GiB.
//   RowsWide: 64-bit addresses per lane; kNoRow reads zero through a masked
//             load.  For inputs of 4 GiB and more (up to 2^31 rows).
constexpr uint32_t kNoRow = 0xFFFFFFFFu;

// A gathered row is named by addr(row) (-1: outside the grid), which the
// kernels stage, then loaded at byte off of the row by load(a, off).
template <int CIN>
struct RowsRaw {
  __amdgpu_buffer_rsrc_t r;
  __device__ __forceinline__ static RowsRaw make(const float* in, uint32_t n_rows) {
    RowsRaw g;
    g.r = input_rsrc(in, n_rows * (uint32_t)(4 * CIN));
    return g;
  }
  __device__ __forceinline__ static uint32_t addr(int row) {
    return row < 0 ? kOutside : (uint32_t)row * (uint32_t)(4 * CIN);
  }
  template <int V>
  __device__ __forceinline__ typename VecT<V>::type load(uint32_t a, uint32_t off) const {
    return gather<V>(r, a + off);
  }
};

template <int CIN>
struct RowsWide {
  const float* base;
  __device__ __forceinline__ static RowsWide make(const float* in, uint32_t) {
    RowsWide g;
    g.base = in;
    return g;
  }
  __device__ __forceinline__ static uint32_t addr(int row) { return row < 0 ? kNoRow : (uint32_t)row; }
  template <int V>
  __device__ __forceinline__ typename VecT<V>::type load(uint32_t row, uint32_t off) const {
    typename VecT<V>::type v;
    if constexpr (V == 1) v = 0.f;
    else v = typename VecT<V>::type(0.f);
    if (row != kNoRow)
      v = *reinterpret_cast<const typename VecT<V>::type*>(base + (uint64_t)row * CIN + (off >> 2));
    return v;
  }
};

template <int V, class G>
__device__ __forceinline__ typename VecT<V>::type gather_at(const G& g, uint32_t a, uint32_t off) {
  return g.template load<V>(a, off);
}

#ifndef OC_UNIT_THREADS
#define OC_UNIT_THREADS 512
#endif
constexpr int kUnitThreads = OC_UNIT_THREADS;

template <int CIN, int NT, int MS, class GP>
__global__ void __launch_bounds__(kUnitThreads) k_conv_unit_mfma(
    int64_t n_leaves, const int32_t* __restrict__ nbt, const int64_t* __restrict__ n_groups,
    const float* __restrict__ in, const float* __restrict__ wm, uint32_t n_rows,
    const float* __restrict__ bias, int cout, int relu, float* __restrict__ out) {
  // Channel blocks: blockIdx.y selects an output block (its weight layout
  // and its [n_leaves][cout] destination).
  wm += (int64_t)blockIdx.y * MfmaCfg<CIN, NT, MS>::WFLOATS;
  out += (int64_t)blockIdx.y * n_leaves * cout;
  if (bias != nullptr) bias += (int64_t)blockIdx.y * cout;
  using C = MfmaCfg<CIN, NT, MS>;
  const GP rin = GP::make(in, n_rows);
  using Vec = typename VecT<C::VEC>::type;
  using Acc = typename AccT<MS>::type;
  extern __shared__ float smem[];
  float* wl = smem;
  int32_t* nb_all = reinterpret_cast<int32_t*>(smem + C::WFLOATS);
  {
    typedef float __attribute__((ext_vector_type(4))) f4;
    const f4* src = reinterpret_cast<const f4*>(wm);
    f4* dst = reinterpret_cast<f4*>(wl);
    for (int i = threadIdx.x; i < C::WFLOATS / 4; i += blockDim.x) dst[i] = src[i];
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // Two neighbourhood tables per wave: the current tile's, and the next
  // tile's, which is staged between the MFMAs of this one.
  int32_t* nb_w = nb_all + wave * (2 * C::GROUPS * 64);
  const int64_t G = min(*n_groups, n_leaves / 8);
  const int64_t n_tiles = (G + C::GROUPS - 1) / C::GROUPS;
  const WaveTiles wt = wave_tiles(n_tiles);
  // Lane roles.
  const int m = lane % MS, g = lane / MS;
  const int gi = m >> 3, o3 = m & 7;
  const int ubase = gi * 64 + ((o3 >> 2) & 1) * 16 + ((o3 >> 1) & 1) * 4 + (o3 & 1);
  const int col = lane % MS;
  // The neighbourhood rows of tile t: loaded from the table (one coalesced
  // load per group) well before they are needed, then written to the LDS
  // table of the wave.
  int32_t tbl[C::GROUPS];
  auto stage_load = [&](int64_t t) {
#pragma unroll
    for (int q = 0; q < C::GROUPS; ++q) {
      const int64_t gidx = t * C::GROUPS + q;
      tbl[q] = (t < wt.end && gidx < G) ? nbt[gidx * 64 + lane] : -1;
    }
  };
  auto stage_rows = [&](int32_t* nbl) {
#pragma unroll
    for (int q = 0; q < C::GROUPS; ++q) nbl[q * 64 + lane] = tbl[q];
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  };
  // The lane's bias values, read once (a load in the epilogue would make it
  // wait for the next tile's gathers as well).
  float bvals[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int co = MS * nt + col;
    bvals[nt] = (bias != nullptr && co < cout) ? bias[co] : 0.f;
  }
  // Epilogue of a finished tile (unit cells need no 1/s^3 scaling).
  auto store_unit_tile = [&](const Acc (&res)[NT], const int32_t* tnb) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int co = MS * nt + col;
      const float bv = bvals[nt];
#pragma unroll
      for (int r = 0; r < (MS == 32 ? 16 : 4); ++r) {
        const int i = MS == 32 ? 8 * (r / 4) + 4 * g + (r % 4) : 4 * g + r;
        const int row0 = tnb[(i >> 3) * 64 + 21];  // voxel (1,1,1): first row of the group
        if (row0 < 0 || row0 + 8 > n_leaves || co >= cout) continue;
        float v = res[nt][r] + bv;
        if (relu & 1) v = fmaxf(v, 0.f);
        out[(int64_t)(row0 + (i & 7)) * cout + co] = v;
      }
    }
  };
  // Software pipeline: the gathered A rows of delta dl+PD and the B operands
  // of delta dl+1 are in flight while the MFMAs of delta dl issue; the
  // gathers of a tile's first PD deltas are issued during the previous
  // tile's last ones (PD + 1 divides 27, so the buffer ring lines up).  The
  // scheduling barriers keep the compiler from sinking the loads back to
  // their use.
  constexpr int PD = unit_prefetch<CIN, MS>();  // deltas of gathers in flight
  static_assert(27 % (PD + 1) == 0, "the gather ring must line up across tiles");
  Vec abuf[PD + 1][C::NV];
  const uint32_t coff = 4u * C::VEC * g;  // the lane's first channel, in bytes
  auto gather_row = [&](uint32_t row, Vec* a) {
#pragma unroll
    for (int v = 0; v < C::NV; ++v) a[v] = gather_at<C::VEC>(rin, row, coff + 4 * C::VSTRIDE * v);
  };
  // The lane's A rows for the first PD deltas of a table.
  uint32_t noff[PD];
  auto first_offsets = [&](const int32_t* t) {
#pragma unroll
    for (int k = 0; k < PD; ++k) noff[k] = GP::addr(t[ubase + (k / 9) * 16 + ((k / 3) % 3) * 4 + k % 3]);
  };
  // A finished tile is stored during the next tile's fifth delta: its stores
  // then queue behind gathers that are already consumed, and the gathers
  // issued after them are consumed deltas later (the memory counter is
  // in issue order).
  Acc pacc[NT];
  const int32_t* pnb = nb_w;
  bool have_prev = false;
  int cur = 0;
  stage_load(wt.first);
  stage_rows(nb_w);
  first_offsets(nb_w);
#pragma unroll
  for (int k = 0; k < PD; ++k) gather_row(noff[k], abuf[k]);
  for (int64_t tile = wt.first; tile < wt.end; tile += wt.stride) {
    int32_t* nb = nb_w + cur * (C::GROUPS * 64);
    int32_t* nb_next = nb_w + (cur ^ 1) * (C::GROUPS * 64);
    const int64_t next = tile + wt.stride;
    // OC_UNIT_ACCS independent accumulator sets (deltas alternate between
    // them) so that consecutive MFMAs do not wait on each other's results.
    constexpr int NA = OC_UNIT_ACCS;
    Acc acc2[NA][NT];
#pragma unroll
    for (int a2 = 0; a2 < NA; ++a2)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int r = 0; r < (MS == 32 ? 16 : 4); ++r) acc2[a2][nt][r] = 0.f;
    Vec bbuf[2][NT][C::NV];
    // The 27 A rows of this lane, read from the table up front so that no
    // LDS round trip sits between a delta's MFMAs and its gathers.
    uint32_t aoff[27];
#pragma unroll
    for (int dl = 0; dl < 27; ++dl) aoff[dl] = GP::addr(nb[ubase + (dl / 9) * 16 + ((dl / 3) % 3) * 4 + dl % 3]);
    auto load_b = [&](int dl, Vec (*b)[C::NV]) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const Vec* bsrc = reinterpret_cast<const Vec*>(wl) + ((dl * NT + nt) * C::NV) * 64 + lane;
#pragma unroll
        for (int v = 0; v < C::NV; ++v) b[nt][v] = bsrc[v * 64];
      }
    };
    load_b(0, bbuf[0]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int dl = 0; dl < 27; ++dl) {
      if (dl + PD < 27) gather_row(aoff[dl + PD], abuf[(dl + PD) % (PD + 1)]);
      else gather_row(noff[dl + PD - 27], abuf[(dl + PD) % (PD + 1)]);  // next tile
      if (dl + 1 < 27) load_b(dl + 1, bbuf[(dl + 1) % 2]);
      // The next tile's neighbourhood rows.
      if (dl == 3) stage_load(next);
      if (dl == 4 && have_prev) store_unit_tile(pacc, pnb);
      if (dl == 18) {
        stage_rows(nb_next);
        first_offsets(nb_next);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int v = 0; v < C::NV; ++v)
#pragma unroll
          for (int e = 0; e < C::VEC; ++e)
            acc2[(v * C::VEC + e) % NA][nt] =
                mfma<MS>(vget<C::VEC>(abuf[dl % (PD + 1)][v], e),
                         vget<C::VEC>(bbuf[dl % 2][nt][v], e), acc2[(v * C::VEC + e) % NA][nt]);
      __builtin_amdgcn_sched_barrier(0);
    }
    Acc acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      acc[nt] = acc2[0][nt];
#pragma unroll
      for (int a2 = 1; a2 < NA; ++a2) acc[nt] += acc2[a2][nt];
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) pacc[nt] = acc[nt];
    pnb = nb;
    have_prev = true;
    cur ^= 1;
    __builtin_amdgcn_wave_barrier();  // nb is rewritten by the next tile
  }
  if (have_prev) store_unit_tile(pacc, pnb);
}

// ---------------------------------------------------------------------------
// MFMA kernels for cells of edge 2, 4 and 8.
//
// A wave takes 16 cells of one edge length SZ and contracts them with
// v_mfma_f32_16x16x4_f32: lane (m = lane % 16, g = lane / 16) feeds CH =
// cin/4 channels of cell m (vector jv: channels VEC (4 jv + g) ..), and the
// weights sit in LDS in the matching B-operand order.  Before they enter the MFMA, the lane builds
// its cell's window sums (origin o):
//   S_delta = x_self * prod_a (SZ - |delta_a|) + sum of x over the one-voxel
//             shell voxels that the window [o+delta, o+delta+SZ) covers,
// one delta_d layer (9 deltas x CH channels) at a time, so that every input
// row a cell needs is gathered at most twice per tile, once per layer that
// reaches it.  The shell geometry of each layer is fixed at compile time, so
// every S_delta stays in a fixed register.
// ---------------------------------------------------------------------------
#ifndef OC_REGION_GROUP
#define OC_REGION_GROUP 3
#endif
#ifndef OC_SHELL_GROUP
#define OC_SHELL_GROUP 8
#endif

template <int CIN, int NT, int MS>
__device__ __forceinline__ void weights_to_lds(const float* __restrict__ wm, float* wl) {
  using C = MfmaCfg<CIN, NT, MS>;
  typedef float __attribute__((ext_vector_type(4))) f4;
  const f4* src = reinterpret_cast<const f4*>(wm);
  f4* dst = reinterpret_cast<f4*>(wl);
  for (int i = threadIdx.x; i < C::WFLOATS / 4; i += blockDim.x) dst[i] = src[i];
  __syncthreads();
}

template <int CIN, int NT>
struct CellCfg {
  using C = MfmaCfg<CIN, NT, 16>;
  static constexpr int CH = C::CH;
  static constexpr int VEC = C::VEC;
  static constexpr int VSTRIDE = C::VSTRIDE;
  static constexpr int NV = C::NV;
  using Vec = typename VecT<VEC>::type;
  using Acc = typename AccT<16>::type;
};

// Channels per lane vector of the 16-row cell kernels.
template <int CIN>
constexpr int cell_vec() {
  return MfmaCfg<CIN, 1, 16>::VEC;
}

// Contract layer JD (deltas 9 JD .. 9 JD + 8) into acc.
template <int CIN, int NT, int JD>
__device__ __forceinline__ void contract_layer(const float (&S)[9][CIN / 4],
                                               const float* wl, int lane,
                                               typename CellCfg<CIN, NT>::Acc (&acc)[NT]) {
  using K = CellCfg<CIN, NT>;
#pragma unroll
  for (int k = 0; k < 9; ++k) {
    const int dl = 9 * JD + k;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int jv = 0; jv < K::NV; ++jv) {
        const typename K::Vec bv =
            reinterpret_cast<const typename K::Vec*>(wl)[((dl * NT + nt) * K::NV + jv) * 64 + lane];
#pragma unroll
        for (int e = 0; e < K::VEC; ++e)
          acc[nt] = mfma<16>(S[k][K::VEC * jv + e], vget<K::VEC>(bv, e), acc[nt]);
      }
    if (k % 3 == 2) __builtin_amdgcn_sched_barrier(0);  // bounds the B loads in flight
  }
}

// The lane's CH channels of row `row`, starting at byte off of the row.
template <int CIN, class G>
__device__ __forceinline__ void gather_channels_at(const G& rin, uint32_t row, uint32_t off,
                                                   float (&x)[CIN / 4]) {
  using K = CellCfg<CIN, 1>;
#pragma unroll
  for (int jv = 0; jv < K::NV; ++jv) {
    const typename K::Vec v = gather_at<K::VEC>(rin, row, off + 4u * K::VSTRIDE * jv);
#pragma unroll
    for (int e = 0; e < K::VEC; ++e) x[K::VEC * jv + e] = vget<K::VEC>(v, e);
  }
}

// The lane's CH channels of the row at byte offset off.
template <int CIN>
__device__ __forceinline__ void gather_channels(__amdgpu_buffer_rsrc_t rin, uint32_t off,
                                                float (&x)[CIN / 4]) {
  using K = CellCfg<CIN, 1>;
#pragma unroll
  for (int jv = 0; jv < K::NV; ++jv) {
    const typename K::Vec v = gather<K::VEC>(rin, off + 4u * K::VSTRIDE * jv);
#pragma unroll
    for (int e = 0; e < K::VEC; ++e) x[K::VEC * jv + e] = vget<K::VEC>(v, e);
  }
}

// The lane's bias values for 16-column tiles (column 16 nt + lane % 16).
template <int NT>
__device__ __forceinline__ void bias16(const float* __restrict__ bias, int cout, int lane,
                                       float (&bv)[NT]) {
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int co = 16 * nt + lane % 16;
    bv[nt] = (bias != nullptr && co < cout) ? bias[co] : 0.f;
  }
}

// Store the tile: D row i (= 4 (lane / 16) + r) belongs to the cell held by
// lane i.
template <int NT>
__device__ __forceinline__ void store_tile16(const typename AccT<16>::type (&acc)[NT], int row,
                                             float inv, int lane, const float (&bvals)[NT],
                                             int cout, int relu, float* __restrict__ out) {
  const int g = lane / 16, col = lane % 16;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int co = 16 * nt + col;
    const float bv = bvals[nt];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int rowi = __shfl(row, 4 * g + r, 64);
      if (rowi < 0 || co >= cout) continue;
      float v = fmaf(acc[nt][r], inv, bv);
      if (relu & 1) v = fmaxf(v, 0.f);
      out[(int64_t)rowi * cout + co] = v;
    }
  }
}

// Range [begin, begin + count) of kind k in the larger-cell list.
__device__ __forceinline__ void kind_range(const int64_t* __restrict__ meta, int kind, int64_t cap,
                                           int64_t& begin, int64_t& count) {
  begin = 0;
  for (int k = 0; k < kind; ++k) begin += meta[k];
  count = meta[kind];
  if (begin > cap) begin = cap;
  if (begin + count > cap) count = cap - begin;
}

// Cell of a list row: sample and global voxel origin (row < 0: none).
__device__ __forceinline__ void cell_origin(const uint64_t* __restrict__ info, int row, int gd,
                                            int gh, int gw, int64_t& n, int (&o)[3]) {
  n = 0;
  o[0] = o[1] = o[2] = 0;
  if (row < 0) return;
  const uint64_t inf = info[row];
  const TreePos p = tree_pos((int64_t)(inf >> 10), gd, gh, gw);
  const Cell c = cell_of((int)(inf & 1023u));
  n = p.n;
  o[0] = 8 * p.d + c.d;
  o[1] = 8 * p.h + c.h;
  o[2] = 8 * p.w + c.w;
}

template <int SZ, int JD, int CH>
__device__ __forceinline__ void init_layer(float (&S)[9][CH], const float (&xs)[CH]) {
  constexpr int fd = SZ - (JD == 1 ? 0 : 1);
#pragma unroll
  for (int k = 0; k < 9; ++k) {
    const float vol = (float)(fd * (SZ - (k / 3 == 1 ? 0 : 1)) * (SZ - (k % 3 == 1 ? 0 : 1)));
#pragma unroll
    for (int e = 0; e < CH; ++e) S[k][e] = xs[e] * vol;
  }
}

// Edge-2 cells.  Shell voxel u (of the 4^3 block [o-1, o+3) minus the cell)
// lies in the window of delta iff u_a - delta_a - 1 is in {0, 1} on every
// axis; layer JD (delta_d = JD - 1) reaches the voxel planes u_d = JD, JD + 1.
// Within a layer the voxels are taken one h-row (u_h = UH) at a time: the
// 8 voxels (u_d in {JD, JD + 1}, u_w = 0..3) of a row are gathered into X,
// and once rows 0..JH+1 are added the window sums of delta-row JH
// (delta_h = JH - 1) are complete and can enter the MFMA while the next
// row's gathers are in flight.
constexpr bool shell2_inner(int u) {
  return (u >> 4) >= 1 && (u >> 4) <= 2 && ((u >> 2) & 3) >= 1 && ((u >> 2) & 3) <= 2 &&
         (u & 3) >= 1 && (u & 3) <= 2;
}

template <int JD, int UH, int K, int CIN>
struct Shell2RowLoad {
  template <class G>
  __device__ __forceinline__ static void run(float (&X)[8][CIN / 4], const uint32_t* rows, const G& rin,
                                             uint32_t choff) {
    constexpr int u = (JD + K / 4) * 16 + UH * 4 + (K % 4);
    if constexpr (!shell2_inner(u)) {
      constexpr int q = shell2_q(u);
      gather_channels_at<CIN>(rin, rows[q], choff, X[K]);
    }
    Shell2RowLoad<JD, UH, K + 1, CIN>::run(X, rows, rin, choff);
  }
};
template <int JD, int UH, int CIN>
struct Shell2RowLoad<JD, UH, 8, CIN> {
  template <class G>
  __device__ __forceinline__ static void run(float (&)[8][CIN / 4], const uint32_t*, const G&, uint32_t) {}
};

// LDS bytes per wave for the shell rows of a 16-cell tile: 57 words per cell
// (56 and a pad, an odd stride, so that the 16 cells' words at one shell
// position fall in different banks).
constexpr int kShell2Stride = 57;
constexpr int kShell2Lds = 16 * kShell2Stride * 4;

// The box sums are separable: the two planes of the row are summed first,
// then neighbouring pairs along w, and each pair sum goes to the two
// delta-rows that reach h-row UH (the cell's own voxels are left out here;
// init_layer counts them).
template <int JD, int UH, int CIN>
__device__ __forceinline__ void shell2_row_add(float (&S)[9][CIN / 4], const float (&X)[8][CIN / 4]) {
  constexpr int CH = CIN / 4;
  float D[4][CH];
#pragma unroll
  for (int uw = 0; uw < 4; ++uw) {
    const bool a = !shell2_inner(JD * 16 + UH * 4 + uw);        // plane JD
    const bool b = !shell2_inner((JD + 1) * 16 + UH * 4 + uw);  // plane JD + 1
#pragma unroll
    for (int e = 0; e < CH; ++e)
      D[uw][e] = a && b ? X[uw][e] + X[4 + uw][e] : (a ? X[uw][e] : (b ? X[4 + uw][e] : 0.f));
  }
#pragma unroll
  for (int jw = 0; jw < 3; ++jw) {
    float P[CH];
#pragma unroll
    for (int e = 0; e < CH; ++e) P[e] = D[jw][e] + D[jw + 1][e];
#pragma unroll
    for (int jh = 0; jh < 3; ++jh) {
      if (UH - jh < 0 || UH - jh > 1) continue;
#pragma unroll
      for (int e = 0; e < CH; ++e) S[jh * 3 + jw][e] += P[e];
    }
  }
}

// Contract delta-row JH (delta_h = JH - 1) of layer JD into acc.
template <int CIN, int NT, int JD, int JH>
__device__ __forceinline__ void contract_row(const float (&S)[9][CIN / 4], const float* wl, int lane,
                                             typename CellCfg<CIN, NT>::Acc (&acc)[NT]) {
  using K = CellCfg<CIN, NT>;
#pragma unroll
  for (int jw = 0; jw < 3; ++jw) {
    const int k = JH * 3 + jw, dl = 9 * JD + k;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int jv = 0; jv < K::NV; ++jv) {
        const typename K::Vec bv =
            reinterpret_cast<const typename K::Vec*>(wl)[((dl * NT + nt) * K::NV + jv) * 64 + lane];
#pragma unroll
        for (int e = 0; e < K::VEC; ++e)
          acc[nt] = mfma<16>(S[k][K::VEC * jv + e], vget<K::VEC>(bv, e), acc[nt]);
      }
  }
}

// As contract_row, for window sums held in the gather layout: the A operand
// of MFMA lane L is fetched from lane perm / 4 (see k_conv_cell2_mfma).
template <int CIN, int NT, int JD, int JH>
__device__ __forceinline__ void contract_row_perm(const float (&S)[9][CIN / 4], const float* wl,
                                                  int lane, int perm,
                                                  typename CellCfg<CIN, NT>::Acc (&acc)[NT]) {
  float P[3][CIN / 4];
#pragma unroll
  for (int jw = 0; jw < 3; ++jw)
#pragma unroll
    for (int e = 0; e < CIN / 4; ++e)
      P[jw][e] = __builtin_bit_cast(
          float, __builtin_amdgcn_ds_bpermute(perm, __builtin_bit_cast(int, S[JH * 3 + jw][e])));
  using K = CellCfg<CIN, NT>;
#pragma unroll
  for (int jw = 0; jw < 3; ++jw) {
    const int dl = 9 * JD + JH * 3 + jw;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int jv = 0; jv < K::NV; ++jv) {
        const typename K::Vec bv =
            reinterpret_cast<const typename K::Vec*>(wl)[((dl * NT + nt) * K::NV + jv) * 64 + lane];
#pragma unroll
        for (int e = 0; e < K::VEC; ++e)
          acc[nt] = mfma<16>(P[jw][K::VEC * jv + e], vget<K::VEC>(bv, e), acc[nt]);
      }
  }
}

// Row steps of the edge-2 window sums, D deep: step K (layer JD = K / 4,
// h-row UH = K % 4) adds its rows, issues the gathers of step K + D, and
// contracts delta-row UH - 1 of the layer once its rows are in; the last
// row of a layer is followed by the next layer's own-voxel terms.
#ifndef OC_CELL2_DEPTH_SMALL
#define OC_CELL2_DEPTH_SMALL 6
#endif
template <int CIN>
constexpr int cell2_depth() {
  return CIN / 4 <= 2 ? OC_CELL2_DEPTH_SMALL : 2;
}

template <int K, int D, int CIN, int NT, class G, int E = 12>
struct Cell2Steps {
  __device__ __forceinline__ static void run(float (&S)[9][CIN / 4], float (&X)[D][8][CIN / 4],
                                             const uint32_t* offm, const G& rin, uint32_t choff,
                                             const float (&xs)[CIN / 4], const float* wl, int lane,
                                             int perm, typename CellCfg<CIN, NT>::Acc (&acc)[NT]) {
    if constexpr (K < E) {
      constexpr int JD = K / 4, UH = K % 4;
      __builtin_amdgcn_sched_barrier(0);
      shell2_row_add<JD, UH, CIN>(S, X[K % D]);
      if constexpr (K + D < 12) {
        Shell2RowLoad<(K + D) / 4, (K + D) % 4, 0, CIN>::run(X[(K + D) % D], offm, rin, choff);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (UH >= 1) contract_row_perm<CIN, NT, JD, UH - 1>(S, wl, lane, perm, acc);
      if constexpr (UH == 3 && JD < 2) {
        __builtin_amdgcn_sched_barrier(0);
        init_layer<2, JD + 1>(S, xs);
      }
      Cell2Steps<K + 1, D, CIN, NT, G, E>::run(S, X, offm, rin, choff, xs, wl, lane, perm, acc);
    }
  }
};

template <int K, int D, int CIN, class G>
struct Cell2Prologue {
  __device__ __forceinline__ static void run(float (&X)[D][8][CIN / 4], const uint32_t* offm, const G& rin,
                                             uint32_t choff) {
    if constexpr (K < D) {
      Shell2RowLoad<K / 4, K % 4, 0, CIN>::run(X[K], offm, rin, choff);
      __builtin_amdgcn_sched_barrier(0);
      Cell2Prologue<K + 1, D, CIN, G>::run(X, offm, rin, choff);
    }
  }
};

// Edge-2 cells.  The window sums are built in a gather layout and moved to
// the MFMA layout before each contraction: in the MFMA layout lane
// m + 16 g holds channel chunk g of cell m, so the 16 lanes that the memory
// pipeline serves together would read 16 different rows; in the gather
// layout lane l holds chunk l % 4 of cell 4 (l / 16) + (l / 4) % 4, so
// those 16 lanes read 4 rows, 64 contiguous bytes each.
// The shell rows come from the parent depth-1 node's 6^3 table (e2key: node
// << 3 | octant, one per cell of the list).
#ifndef OC_CELL2_THREADS
#define OC_CELL2_THREADS 512
#endif
constexpr int kMfmaThreads = OC_CELL2_THREADS;

template <int CIN, int NT, class GP>
__global__ void __launch_bounds__(kMfmaThreads) k_conv_cell2_mfma(
    int64_t n_leaves, const int32_t* __restrict__ brow, const int32_t* __restrict__ e2key,
    const int32_t* __restrict__ ntab, int64_t ncap, const int64_t* __restrict__ meta,
    const float* __restrict__ in, const float* __restrict__ wm, uint32_t n_rows,
    const float* __restrict__ bias, int cout, int relu, float* __restrict__ out) {
  // Channel blocks: blockIdx.y selects an output block (its weight layout
  // and its [n_leaves][cout] destination).
  wm += (int64_t)blockIdx.y * MfmaCfg<CIN, NT, 16>::WFLOATS;
  out += (int64_t)blockIdx.y * n_leaves * cout;
  if (bias != nullptr) bias += (int64_t)blockIdx.y * cout;
  using K = CellCfg<CIN, NT>;
  constexpr int CH = K::CH;
  extern __shared__ float smem[];
  float* wl = smem;
  weights_to_lds<CIN, NT, 16>(wm, wl);
  const GP rin = GP::make(in, n_rows);
  const int lane = threadIdx.x & 63;
  int64_t lbeg, lcnt;
  kind_range(meta, 3, n_leaves, lbeg, lcnt);
  const WaveTiles wt = wave_tiles((lcnt + 15) / 16);
  // Gather layout: cell cl, chunk q.  MFMA lane (m, g) takes its operands
  // from lane 16 (m / 4) + 4 (m % 4) + g.
  const int cl = 4 * (lane >> 4) + ((lane >> 2) & 3), q = lane & 3;
  const int perm = 4 * (16 * ((lane & 15) >> 2) + 4 * (lane & 3) + (lane >> 4));
  const uint32_t choff = 4u * (uint32_t)(K::VEC * q);  // the lane's first channel
  float bvals[NT];
  bias16<NT>(bias, cout, lane, bvals);
  // The wave's shell offsets: 56 per cell, after the weights.
  uint32_t* offm = reinterpret_cast<uint32_t*>(smem + MfmaCfg<CIN, NT, 16>::WFLOATS) +
                   (threadIdx.x >> 6) * (kShell2Lds / 4) + cl * kShell2Stride;
  // Tiles are pipelined: a tile's row and key are loaded at the start of
  // the tile before it, and its shell table entries halfway through that
  // tile's row steps, so that a tile starts with its shell rows at hand.
  // Row and key of the lane's cell of `tile` (row -1: no cell).
  auto cell_of_tile = [&](int64_t tile, int& row, int32_t& key) {
    const int64_t idx = tile * 16 + cl;
    const bool in = tile < wt.end && idx < lcnt;
    row = in ? brow[lbeg + idx] : -1;
    key = in ? e2key[idx] : 0;
  };
  // The lane's 14 shell table entries (chunk q takes shell voxels 4 j + q of
  // its cell; the cell's 4^3 neighbourhood is the sub-block of its node's
  // table at twice its octant).
  auto shell_entries = [&](int& row, int32_t key, int (&mine)[14]) {
    const int64_t node = key >> 3;
    if (row >= n_leaves || key < 0 || node >= ncap) row = -1;  // only a non-canonical structure
    const int o2 = key & 7;
    // Read whatever the cell (node 0's entries when there is none, taken by
    // no one), so that the loads need no branch; with no node at all there
    // are no edge-2 cells and nothing is read.
    const int32_t* nt = ntab + (row >= 0 ? node : 0) * kNodeEntries + 2 * ((o2 >> 2) & 1) * 36 +
                        2 * ((o2 >> 1) & 1) * 6 + 2 * (o2 & 1);
#pragma unroll
    for (int j = 0; j < 14; ++j) {
      const int u = c_shell2.u[4 * j + q];
      mine[j] = ncap > 0 ? nt[(u >> 4) * 36 + ((u >> 2) & 3) * 6 + (u & 3)] : -1;
    }
  };
  int row_n;
  int32_t key_n;
  int mine_n[14];
  cell_of_tile(wt.first, row_n, key_n);
  shell_entries(row_n, key_n, mine_n);
  for (int64_t tile = wt.first; tile < wt.end; tile += wt.stride) {
    int row = row_n;
    // Shell rows of this tile, in the wave's LDS area.
#pragma unroll
    for (int j = 0; j < 14; ++j) offm[4 * j + q] = GP::addr(row >= 0 ? mine_n[j] : -1);
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    cell_of_tile(tile + wt.stride, row_n, key_n);
    float xs[CH];
    gather_channels_at<CIN>(rin, GP::addr(row), choff, xs);
    typename K::Acc acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[nt][r] = 0.f;
    // The 12 row steps (layer JD, h-row UH) run D deep: the gathers of step
    // k + D are issued once step k's rows are added (D = 2, or 6 where a
    // lane's row piece is at most 2 floats).
    constexpr int D = cell2_depth<CIN>();
    float S[9][CH];
    float X[D][8][CH];
    init_layer<2, 0>(S, xs);
    Cell2Prologue<0, D, CIN, GP>::run(X, offm, rin, choff);
    Cell2Steps<0, D, CIN, NT, GP, 6>::run(S, X, offm, rin, choff, xs, wl, lane, perm, acc);
    shell_entries(row_n, key_n, mine_n);  // the next tile's
    Cell2Steps<6, D, CIN, NT, GP>::run(S, X, offm, rin, choff, xs, wl, lane, perm, acc);
    __builtin_amdgcn_wave_barrier();  // offm is rewritten by the next tile
    // The row of cell m, for the store's MFMA layout.
    const int row_m = __builtin_amdgcn_ds_bpermute(perm, row);
    store_tile16<NT>(acc, row_m, (relu & 2) ? 1.f : 0.125f, lane, bvals, cout, relu, out);
  }
}

// ---------------------------------------------------------------------------
// Boundary sums.  Boundary set e (e in {-1, 0, 1}^3, e != 0) of an aligned
// cubic block holds the voxels whose coordinate along every axis with
// e_a != 0 is the block's first (e_a = -1) or last (e_a = +1): 6 faces, 12
// edge lines and 8 corners.  Once per convolution the input is summed over
// every boundary set of every split tree and every split depth-1 node, per
// voxel (a leaf counts once for each of its voxels in the set).  A split
// tree t owns slot sbase[t] and, for its k-th split depth-1 node, slot
// sbase[t] + 1 + k; slot s holds 26 rows of cin floats at
// bsum[(26 s + set) cin].
// ---------------------------------------------------------------------------
constexpr int kSets = 26;

__host__ __device__ constexpr int bset(int ed, int eh, int ew) {
  return (ed + 1) * 9 + (eh + 1) * 3 + (ew + 1) - ((ed + 1) * 9 + (eh + 1) * 3 + (ew + 1) > 13);
}

// Is coordinate x (of a block of edge B) inside set component e?
__host__ __device__ constexpr bool in_set(int e, int x, int B) {
  return e == 0 || (e < 0 ? x == 0 : x == B - 1);
}

// The 56 boundary voxels V (= 16 x0 + 4 x1 + x2) of a 4^3 block, K-th in
// ascending order: load reads each from its leaf (a2: gather address of each
// 2^3 octant's leaf or first unit voxel, st2: the address step from one unit
// voxel of the octant to the next, 0 for an unsplit octant), add puts each
// into the sets that hold it.
constexpr bool interior4(int v) {
  return (v >> 4) % 3 != 0 && ((v >> 2) & 3) % 3 != 0 && (v & 3) % 3 != 0;
}

// The boundary sets (26-bit mask over the set index) that hold voxel V of a
// 4^3 block.
constexpr uint32_t voxel_sets(int V) {
  uint32_t m = 0;
  for (int r = 0; r < 27; ++r)
    if (r != 13 && in_set(r / 9 - 1, V >> 4, 4) && in_set((r / 3) % 3 - 1, (V >> 2) & 3, 4) &&
        in_set(r % 3 - 1, V & 3, 4))
      m |= 1u << (r - (r > 13));
  return m;
}

template <int V, int K>
struct BoundaryVoxels {
  static constexpr int x0 = V >> 4, x1 = (V >> 2) & 3, x2 = V & 3;
  static constexpr bool skip = interior4(V);
  static constexpr int NK = skip ? K : K + 1;
  // need: the sets that are read; a voxel in none of them reads zero (no
  // memory traffic) and the sets it would change are not written.
  template <int CIN, class G>
  __device__ __forceinline__ static void load(float (&xv)[56], const uint32_t (&a2)[8], const uint32_t (&st2)[8],
                                              const G& rin, uint32_t off, uint32_t need) {
    if constexpr (!skip) {
      constexpr int o2 = 4 * (x0 >> 1) + 2 * (x1 >> 1) + (x2 >> 1);
      constexpr uint32_t u = 4 * (x0 & 1) + 2 * (x1 & 1) + (x2 & 1);
      const uint32_t a = (need & voxel_sets(V)) != 0u ? a2[o2] + u * st2[o2] : G::addr(-1);
      xv[K] = gather_at<1>(rin, a, off);
    }
    BoundaryVoxels<V + 1, NK>::template load<CIN, G>(xv, a2, st2, rin, off, need);
  }
  __device__ __forceinline__ static void add(float (&cs)[kSets], const float (&xv)[56]) {
    if constexpr (!skip) {
#pragma unroll
      for (int r = 0; r < 27; ++r) {
        if (r == 13) continue;
        if (in_set(r / 9 - 1, x0, 4) && in_set((r / 3) % 3 - 1, x1, 4) && in_set(r % 3 - 1, x2, 4))
          cs[r - (r > 13)] += xv[K];
      }
    }
    BoundaryVoxels<V + 1, NK>::add(cs, xv);
  }
};
template <int K>
struct BoundaryVoxels<64, K> {
  template <int CIN, class G>
  __device__ __forceinline__ static void load(float (&)[56], const uint32_t (&)[8], const uint32_t (&)[8], const G&,
                                              uint32_t, uint32_t) {}
  __device__ __forceinline__ static void add(float (&)[kSets], const float (&)[56]) {}
};

// The boundary sets of a tree that its depth-1 child o1 touches (26-bit mask
// over the set index): along each axis a set with e_a = -1 holds the children
// with coordinate bit 0, e_a = +1 those with bit 1, e_a = 0 all of them.
template <int A, int E>
__host__ __device__ constexpr uint32_t sets_with_dir() {
  uint32_t m = 0;
  for (int r = 0; r < 27; ++r) {
    const int e = A == 0 ? r / 9 - 1 : (A == 1 ? (r / 3) % 3 - 1 : r % 3 - 1);
    if (r != 13 && e == E) m |= 1u << (r - (r > 13));
  }
  return m;
}

__device__ __forceinline__ uint32_t child_sides(int o1) {
  const uint32_t miss_d = (o1 & 4) ? sets_with_dir<0, -1>() : sets_with_dir<0, 1>();
  const uint32_t miss_h = (o1 & 2) ? sets_with_dir<1, -1>() : sets_with_dir<1, 1>();
  const uint32_t miss_w = (o1 & 1) ? sets_with_dir<2, -1>() : sets_with_dir<2, 1>();
  return ((1u << kSets) - 1u) & ~(miss_d | miss_h | miss_w);
}

// Voxels of an unsplit depth-1 child (4^3) in a tree set that it touches:
// 4 per axis along which the set spans the tree, 1 across it.
__host__ __device__ constexpr float child_set_voxels(int s) {
  const int r = s + (s >= 13);
  return (float)((r / 9 == 1 ? 4 : 1) * ((r / 3) % 3 == 1 ? 4 : 1) * (r % 3 == 1 ? 4 : 1));
}

// Position of the k-th set bit of m (k < popcount(m)).
__device__ __forceinline__ int nth_bit(uint32_t m, int k) {
  for (int i = 0; i < k; ++i) m &= m - 1u;
  return __ffs(m) - 1;
}

// Split trees per wave of the boundary sums.
constexpr int sum_trees_per_wave(int cin) { return 64 / cin > 8 ? 64 / cin / 8 : 1; }

// One split tree per wave (two per wave for CIN = 4), split into lane
// groups of CIN lanes (lane = channel).  The groups take the tree's split
// depth-1 children in turn: each is summed from its 56 boundary voxels, each
// read from the leaf that holds it, all 56 loads in flight before the sums.
// An unsplit child is one leaf, so its share of a tree set is its row times
// its voxels in the set.  A tree set is the sum of the same set over the
// children on that side: each group sums its children, then the groups of
// the tree add theirs (a fixed butterfly, so the result is deterministic).
template <int CIN, class GP>
__global__ void __launch_bounds__(256) k_boundary_sums(
    const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix,
    const int32_t* __restrict__ stl, const int64_t* __restrict__ meta,
    const int64_t* __restrict__ sbase, int64_t n_trees, int64_t cap, const float* __restrict__ in,
    uint32_t n_rows, float* __restrict__ bsum, const int64_t* __restrict__ p8t,
    const int64_t* __restrict__ p8n, int64_t t0, int64_t t1, const uint32_t* __restrict__ smask) {
  constexpr int NG = 64 / CIN;              // lane groups per wave
  constexpr int TPW = sum_trees_per_wave(CIN);
  constexpr int GPT = NG / TPW;             // lane groups per tree
  const int lane = threadIdx.x & 63, c = lane % CIN, grp = lane / CIN;
  const int sub = grp / GPT, gi = grp % GPT;
  int64_t n_split = n_trees - meta[0] - meta[1];
  n_split = n_split < 0 ? 0 : (n_split > n_trees ? n_trees : n_split);
  // The split trees among trees [t0, t1): list entries [j0, j1).
  const int64_t j0 = min(n_split, max((int64_t)0, t0 - p8t[t0] - p8n[t0]));
  const int64_t j1 = min(n_split, max(j0, t1 - p8t[t1] - p8n[t1]));
  const GP rin = GP::make(in, n_rows);
  const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t j = j0 + wave * TPW + sub; j < j1; j += nwaves * TPW) {
    const int64_t t = stl[j];
    const Bits b = load_bits(trees, t);
    const int rbase = (int)prefix[t];
    const int64_t s0 = sbase[t];
    const uint32_t m1 = (uint32_t)(b.lo >> 1) & 0xFFu;  // split depth-1 children
    const int p1 = __popc(m1);
    // Eq. 3 for the depth-2 nodes below a split child o1 and for the first
    // unit voxel of each split one, from the set-bit counts below bit 1 + o1,
    // below bit 9 + 8 o1 + o2 and of the whole string.  Bit j of dbits is
    // split bit 9 + j (the depth-2 nodes).
    const uint64_t dbits = (b.lo >> 9) | ((uint64_t)b.hi << 55);
    const int pall = popc_all(b), p9 = __popcll(b.lo & 0x1FFull);
    // The gather address of a row: a2 holds the channel offset for the raw
    // policy, the wide one takes it at the load.
    constexpr bool RAW = std::is_same<GP, RowsRaw<CIN>>::value;
    const uint32_t coff = RAW ? 4u * c : 0u, loff = RAW ? 0u : 4u * c;
    const uint32_t step = RAW ? 4u * CIN : 1u;  // address step of one row
    float ts[kSets];
#pragma unroll
    for (int s = 0; s < kSets; ++s) ts[s] = 0.f;
    for (int k = gi; k < p1; k += GPT) {
      const int o1 = nth_bit(m1, k);
      const uint32_t sp = (uint32_t)(dbits >> (8 * o1)) & 0xFFu;  // split octants
      const int pd1 = __popcll(b.lo & ((2ull << o1) - 1ull));
      const int pd2 = p9 + __popcll(dbits & ((1ull << (8 * o1)) - 1ull));
      uint32_t a2[8], st2[8];
#pragma unroll
      for (int o2 = 0; o2 < 8; ++o2) {
        const int p2 = pd2 + __popc(sp & ((1u << o2) - 1u));
        const bool s2 = (sp >> o2) & 1u;
        const int row = rbase + (s2 ? 8 * p2 + 1 - pall : 8 * pd1 + 1 - p2 + o2);
        a2[o2] = GP::addr(row) + coff;
        st2[o2] = s2 && row >= 0 ? step : 0u;
      }
      // The child's sets that are read: its own, and those of the tree's
      // sets on its side.
      const int64_t slot = s0 + 1 + k;
      const uint32_t mk = slot < cap ? smask[slot] : 0u;
      const uint32_t need = mk | (s0 < cap ? smask[s0] & child_sides(o1) : 0u);
      float xv[56];
      BoundaryVoxels<0, 0>::load<CIN, GP>(xv, a2, st2, rin, loff, need);
      __builtin_amdgcn_sched_barrier(0);
      float cs[kSets];
#pragma unroll
      for (int s = 0; s < kSets; ++s) cs[s] = 0.f;
      BoundaryVoxels<0, 0>::add(cs, xv);
      if (slot < cap) {
        float* dst = bsum + slot * (kSets * CIN) + c;
#pragma unroll
        for (int s = 0; s < kSets; ++s)
          if ((mk >> s) & 1u) dst[s * CIN] = cs[s];
      }
      const uint32_t side = child_sides(o1);
#pragma unroll
      for (int s = 0; s < kSets; ++s)
        if ((side >> s) & 1u) ts[s] += cs[s];
    }
    const uint32_t u1 = ~m1 & 0xFFu;  // unsplit depth-1 children (leaves)
    for (int k = gi; k < 8 - p1; k += GPT) {
      const int o1 = nth_bit(u1, k);
      const float x = gather_at<1>(rin, GP::addr(rbase + data_idx(b, 1 + o1)), 4u * c);
      const uint32_t side = child_sides(o1);
#pragma unroll
      for (int s = 0; s < kSets; ++s)
        if ((side >> s) & 1u) ts[s] = fmaf(child_set_voxels(s), x, ts[s]);
    }
#pragma unroll
    for (int off = CIN; off < CIN * GPT; off <<= 1)
#pragma unroll
      for (int s = 0; s < kSets; ++s) ts[s] += __shfl_xor(ts[s], off, 64);
    if (gi == 0 && s0 < cap) {
      const uint32_t mk = smask[s0];
      float* dst = bsum + s0 * (kSets * CIN) + c;
#pragma unroll
      for (int s = 0; s < kSets; ++s)
        if ((mk >> s) & 1u) dst[s * CIN] = ts[s];
    }
  }
}

__global__ void k_zero_u32(uint32_t* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

// Region codes of the edge-4 and edge-8 cells (structure only, built once per
// structure; bkey gives each entry's tree and bit index).  For list entry j
// (the first three kinds) and shell region r
// (the 27 offsets dir without the centre, r = index of dir minus one past
// the centre), codes[r ccap + j] = the row of the leaf that covers the
// neighbouring block at offset dir (the tree for an edge-8 cell, the depth-1
// node for an edge-4 one), -2 - s if that block is split and has
// boundary-sum slot s, -1 outside the grid.  A corner region is one voxel,
// so its code is always the row of the leaf that holds that voxel.  smask[s]
// collects the boundary sets of slot s that some cell reads.
__global__ void k_region_codes(const uint32_t* __restrict__ trees,
                               const int64_t* __restrict__ prefix, int gd, int gh, int gw,
                               int64_t n_leaves, const int64_t* __restrict__ bkey,
                               const int32_t* __restrict__ brow, const int64_t* __restrict__ meta,
                               const int64_t* __restrict__ sbase, int64_t cap, int64_t ccap,
                               int32_t* __restrict__ codes, uint32_t* __restrict__ smask) {
  int64_t n8 = meta[0] + meta[1], nbig = n8 + meta[2];
  if (nbig > ccap) nbig = ccap;
  if (nbig > n_leaves) nbig = n_leaves;
  // Grid-stride over the cells (their count is on the device).
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nbig;
       j += (int64_t)gridDim.x * blockDim.x) {
  const int sz = j < n8 ? 8 : 4;
  int row = brow[j];
  if (row >= n_leaves) row = -1;  // only a non-canonical structure gets here
  int64_t n = 0;
  int o[3] = {0, 0, 0};
  if (row >= 0) {
    const int64_t k = bkey[j];
    const TreePos p = tree_pos(k >> 10, gd, gh, gw);
    const Cell c = cell_of((int)(k & 1023));
    n = p.n;
    o[0] = 8 * p.d + c.d;
    o[1] = 8 * p.h + c.h;
    o[2] = 8 * p.w + c.w;
  }
  const int lim[3] = {8 * gd, 8 * gh, 8 * gw};
  // Region r's block: its tree tt (-1 outside the grid) and its corner lo.
  auto locate = [&](int r, int (&lo)[3]) -> int64_t {
    const int dir[3] = {r / 9 - 1, (r / 3) % 3 - 1, r % 3 - 1};
    bool inside = row >= 0;
    for (int a = 0; a < 3; ++a) {
      lo[a] = dir[a] < 0 ? o[a] - 1 : (dir[a] == 0 ? o[a] : o[a] + sz);
      const int hi = dir[a] < 0 ? o[a] : (dir[a] == 0 ? o[a] + sz : o[a] + sz + 1);
      inside = inside && lo[a] >= 0 && hi <= lim[a];
    }
    return inside ? ((n * gd + (lo[0] >> 3)) * gh + (lo[1] >> 3)) * gw + (lo[2] >> 3) : -1;
  };
  // Region r's code from its tree's words, first row and slot base.
  auto resolve = [&](int r, const int (&lo)[3], int64_t tt, const uint4 tw, int64_t rr, int64_t sb) {
    const int dir[3] = {r / 9 - 1, (r / 3) % 3 - 1, r % 3 - 1};
    int32_t code = -1;
    if (tt >= 0) {
      const uint32_t w0 = tw.x;  // split bits 0..31
      int64_t slot = -1;
      const bool corner = dir[0] != 0 && dir[1] != 0 && dir[2] != 0;
      if (corner) {
        Bits b;
        b.lo = (uint64_t)tw.x | ((uint64_t)tw.y << 32);
        b.hi = tw.z & 0x1FFu;
        rr += data_idx(b, leaf_at(b, lo[0] & 7, lo[1] & 7, lo[2] & 7));
      } else if (w0 & 1u) {
        if (sz == 8) {
          slot = sb;
        } else {
          const int o1 = 4 * ((lo[0] >> 2) & 1) + 2 * ((lo[1] >> 2) & 1) + ((lo[2] >> 2) & 1);
          const int m = __popc((w0 >> 1) & ((1u << o1) - 1u));  // split depth-1 nodes before it
          if ((w0 >> (1 + o1)) & 1u) slot = sb + 1 + m;
          else rr += o1 - m;  // Eq. 3 for a depth-1 leaf
        }
      }
      if (slot >= 0) code = slot < cap && slot < 0x7FFFFFF0LL ? (int32_t)(-2 - slot) : -1;
      if (code <= -2) {
        // The sets a cell reads for region dir: e_a = -dir_a where dir_a != 0,
        // any value on the other axes.
        uint32_t mk = 0;
        for (int q = 0; q < 27; ++q) {
          if (q == 13) continue;
          const int e3[3] = {q / 9 - 1, (q / 3) % 3 - 1, q % 3 - 1};
          if ((dir[0] == 0 || e3[0] == -dir[0]) && (dir[1] == 0 || e3[1] == -dir[1]) &&
              (dir[2] == 0 || e3[2] == -dir[2]))
            mk |= 1u << (q - (q > 13));
        }
        atomicOr(&smask[slot], mk);
      }
      else code = rr < n_leaves ? (int32_t)rr : -1;  // only a non-canonical structure exceeds
    }
    codes[(int64_t)(r - (r > 13)) * ccap + j] = code;
  };
  if (gridDim.y == 1) {
    // One thread per cell: the regions in two groups of 13, each group's
    // tree words, first rows and slot bases loaded together (a region
    // outside the grid reads tree 0's), then resolved.
#pragma unroll
    for (int g0 = 0; g0 < kSets; g0 += 13) {
      int lo[13][3];
      int64_t tt[13], rr[13], sb[13];
      uint4 tw[13];
#pragma unroll
      for (int i = 0; i < 13; ++i) {
        const int rs = g0 + i, r = rs + (rs >= 13 ? 1 : 0);
        tt[i] = locate(r, lo[i]);
        const int64_t q = tt[i] >= 0 ? tt[i] : 0;
        tw[i] = reinterpret_cast<const uint4*>(trees)[q];
        rr[i] = prefix[q];
        sb[i] = sbase[q];
      }
#pragma unroll
      for (int i = 0; i < 13; ++i) {
        const int rs = g0 + i, r = rs + (rs >= 13 ? 1 : 0);
        resolve(r, lo[i], tt[i], tw[i], rr[i], sb[i]);
      }
    }
  } else {
    // Grid row y takes regions y, y + gridDim.y, ... (indices without the
    // centre): on small structures one region per thread, so that a cell's
    // lookups run side by side.
    for (int rs = (int)blockIdx.y; rs < kSets; rs += (int)gridDim.y) {
      const int r = rs + (rs >= 13 ? 1 : 0);
      int lo[3];
      const int64_t t = locate(r, lo);
      const int64_t q = t >= 0 ? t : 0;
      resolve(r, lo, t, reinterpret_cast<const uint4*>(trees)[q], prefix[q], sbase[q]);
    }
  }
  }
}

// ---------------------------------------------------------------------------
// Neighbourhood tables of a preparation (structure only), one wave per split
// tree at a time (grid-stride over the split-tree list).  The 27 trees
// around the wave's tree (bits, first row) are read once into LDS; every
// table entry is then resolved from that copy (the voxel's leaf by the
// tree's split bits, its row by Eq. 3), without branches and without
// further global loads:
//   - ntab: for every split depth-1 node (index d1pre[tree] + k for the
//     tree's k-th), the rows of the 6^3 voxels [o - 1, o + 5) around its 4^3
//     block, -1 outside the grid.  The 4^3 neighbourhood of each of its
//     depth-2 octants (a unit-voxel group or an edge-2 cell) is the sub-block
//     at twice the octant's offset.
//   - nbt: those sub-blocks of the unit-voxel groups, 64 rows per group in
//     group order, the layout the unit-voxel kernel stages.
// ---------------------------------------------------------------------------
struct NbTree {
  uint32_t w0;      // split bits 0..31 (the root's and the depth-1 nodes' are 0..8)
  uint32_t d0, d1;  // depth-2 split bits: bit j of (d1, d0) is bit 9 + j
  int32_t p9;       // set bits among 0..8
  int32_t pd0;      // p9 + set bits of d0
  int32_t pall;     // set bits among 0..72
  uint32_t row0;    // first row (prefix), modulo 2^32
  int32_t lim;      // n_leaves - first row, clamped to int32 (INT32_MIN outside the grid)
};

// Row of the leaf holding voxel (d, h, w), local coordinates of the wave's
// tree in [-1, 8]; -1 outside the grid or past n_leaves (non-canonical).
// The neighbour tree along an axis is (x + 8) >> 3 (0 below, 1 the wave's
// own, 2 above), and the octant bits of x & 7 are those of x itself.  The
// leaf's offset is Eq. 3 at the depth where the descent stops, from the
// set-bit counts below bits 1 + o1 and 9 + 8 o1 + o2 (the depth-1 and
// depth-2 node bits) and of the whole string; an unsplit root is the only
// leaf (offset 0).
__device__ __forceinline__ int32_t nb_voxel_row(const NbTree* __restrict__ nt, int d, int h, int w) {
  const NbTree n = nt[((d + 8) >> 3) * 9 + ((h + 8) >> 3) * 3 + ((w + 8) >> 3)];
  const int o1 = (((d >> 2) & 1) << 2) | (((h >> 2) & 1) << 1) | ((w >> 2) & 1);
  const int o2 = (((d >> 1) & 1) << 2) | (((h >> 1) & 1) << 1) | ((w >> 1) & 1);
  const int o3 = ((d & 1) << 2) | ((h & 1) << 1) | (w & 1);
  const int p1 = __popc(n.w0 & ((2u << o1) - 1u));  // bits 0 .. o1
  const uint32_t s1 = (n.w0 >> (1 + o1)) & 1u;
  const int jj = ((o1 & 3) << 3) | o2;  // bit 9 + 8 o1 + o2, within d0 or d1
  const uint32_t dw = o1 < 4 ? n.d0 : n.d1;
  const int p2 = (o1 < 4 ? n.p9 : n.pd0) + __popc(dw & ((1u << jj) - 1u));
  const uint32_t s2 = (dw >> jj) & 1u;
  const int di1 = 1 - p1 + o1, di2 = 8 * p1 + 1 - p2 + o2, di3 = 8 * p2 + 1 - n.pall + o3;
  const int di = (n.w0 & 1u) ? (s1 ? (s2 ? di3 : di2) : di1) : 0;
  return di < n.lim ? (int32_t)(n.row0 + (uint32_t)di) : -1;
}

constexpr int kTreeWaves = 4;
#ifndef OC_TREE_TABLE_BLOCKS
#define OC_TREE_TABLE_BLOCKS 16
#endif

__global__ void __launch_bounds__(64 * kTreeWaves) k_tree_tables(
    const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix, int gd, int gh, int gw,
    int64_t n_trees, int64_t n_leaves, const int32_t* __restrict__ stl, const int64_t* __restrict__ meta,
    const int64_t* __restrict__ gpre, const int64_t* __restrict__ d1pre, int32_t* __restrict__ nbt,
    int64_t gcap, int32_t* __restrict__ ntab, int64_t ncap) {
  __shared__ NbTree s_nb[kTreeWaves][27];
  __shared__ int32_t s_node[kTreeWaves][kNodeEntries];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int64_t n_split = n_trees - meta[0] - meta[1];
  n_split = n_split < 0 ? 0 : (n_split > n_trees ? n_trees : n_split);
  NbTree* nb = s_nb[wave];
  int32_t* sn = s_node[wave];
  // The 6^3 block coordinates of the lane's entries lane + 64 k.
  int ud[4], uh[4], uw[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int u = lane + 64 * k;
    ud[k] = u / 36;
    uh[k] = (u / 6) % 6;
    uw[k] = u % 6;
  }
  const int64_t nwaves = (int64_t)gridDim.x * kTreeWaves;
  for (int64_t j = (int64_t)blockIdx.x * kTreeWaves + wave; j < n_split; j += nwaves) {
    const int64_t t = stl[j];
    if (lane < 27) {
      const TreePos p = tree_pos(t, gd, gh, gw);
      const int qd = p.d + lane / 9 - 1, qh = p.h + (lane / 3) % 3 - 1, qw = p.w + lane % 3 - 1;
      uint32_t w0 = 0u, w1 = 0u, w2 = 0u;
      int64_t r0 = 0, lim = INT32_MIN;
      if (qd >= 0 && qh >= 0 && qw >= 0 && qd < gd && qh < gh && qw < gw) {
        const int64_t q = ((p.n * gd + qd) * gh + qh) * gw + qw;
        const uint4 wv = reinterpret_cast<const uint4*>(trees)[q];
        w0 = wv.x;
        w1 = wv.y;
        w2 = wv.z & 0x1FFu;
        r0 = prefix[q];
        lim = n_leaves - r0;
        lim = lim < INT32_MIN ? INT32_MIN : (lim > INT32_MAX ? INT32_MAX : lim);
      }
      NbTree n;
      n.w0 = w0;
      n.d0 = (w0 >> 9) | (w1 << 23);
      n.d1 = (w1 >> 9) | (w2 << 23);
      n.p9 = __popc(w0 & 0x1FFu);
      n.pd0 = n.p9 + __popc(n.d0);
      n.pall = __popc(w0) + __popc(w1) + __popc(w2);
      n.row0 = (uint32_t)r0;
      n.lim = (int32_t)lim;
      nb[lane] = n;
    }
    // The wave's own bits and counters, wave-uniform.
    const uint4 ow = reinterpret_cast<const uint4*>(trees)[t];
    const uint32_t b0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)ow.x);
    const uint32_t b1 = (uint32_t)__builtin_amdgcn_readfirstlane((int)ow.y);
    const uint32_t b2 = (uint32_t)__builtin_amdgcn_readfirstlane((int)ow.z);
    int64_t g = gpre[t], node = d1pre[t];
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
#pragma unroll 1  // rolled: fewer registers, more waves in flight
    for (int o1 = 0; o1 < 8; ++o1) {
      if (!((b0 >> (1 + o1)) & 1u)) continue;
      const int od = 4 * ((o1 >> 2) & 1) - 1, oh = 4 * ((o1 >> 1) & 1) - 1, ow1 = 4 * (o1 & 1) - 1;
      int32_t v[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        v[k] = lane + 64 * k < kNodeEntries ? nb_voxel_row(nb, od + ud[k], oh + uh[k], ow1 + uw[k]) : -1;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int u = lane + 64 * k;
        if (u < kNodeEntries) {
          sn[u] = v[k];
          if (node < ncap) ntab[node * kNodeEntries + u] = v[k];
        }
      }
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "workgroup");
      for (int o2 = 0; o2 < 8; ++o2) {
        const int n2 = 9 + 8 * o1 + o2;
        if (!(((n2 < 32 ? b0 : (n2 < 64 ? b1 : b2)) >> (n2 & 31)) & 1u)) continue;
        const int idx = (2 * ((o2 >> 2) & 1) + (lane >> 4)) * 36 + (2 * ((o2 >> 1) & 1) + ((lane >> 2) & 3)) * 6 +
                        2 * (o2 & 1) + (lane & 3);
        if (g < gcap) nbt[g * 64 + lane] = sn[idx];
        ++g;
      }
      ++node;
      __builtin_amdgcn_wave_barrier();  // sn is rewritten for the next node
    }
    __builtin_amdgcn_wave_barrier();  // nb is rewritten for the next tree
  }
}

// Edge-4 and edge-8 cells.  The shell splits into 26 regions (faces, edges,
// corners).  Region dir lies in the neighbouring block at offset dir (a
// tree for SZ = 8, a depth-1 node for SZ = 4) and is that block's boundary
// set -dir.  Along an axis with dir_a != 0 it lies in the window of delta
// only for delta_a = dir_a; along the others it spans the cell, and the
// window cuts off its last voxel plane (delta_a = -1) or its first
// (delta_a = +1).  If one leaf covers the block, the region adds that leaf's
// row times the number of its voxels in the window; otherwise the block's
// boundary sums give it by inclusion-exclusion: set -dir, minus for each cut
// axis the set that also fixes that axis to the cut side, plus the sets that
// fix two or three cut axes.  Layer JD takes the regions with dir_d in
// {0, JD - 1}.
template <int R, int JD, int SZ, int CH>
__device__ __forceinline__ void region_add(float (&S)[9][CH], const float (&x)[CH]) {
  constexpr int dir0 = R / 9 - 1, dir1 = (R / 3) % 3 - 1, dir2 = R % 3 - 1;
#pragma unroll
  for (int j1 = 0; j1 < 3; ++j1) {
    if (dir1 != 0 && j1 != dir1 + 1) continue;
#pragma unroll
    for (int j2 = 0; j2 < 3; ++j2) {
      if (dir2 != 0 && j2 != dir2 + 1) continue;
      const float wgt = (float)((dir0 == 0 ? SZ - (JD != 1) : 1) * (dir1 == 0 ? SZ - (j1 != 1) : 1) *
                                (dir2 == 0 ? SZ - (j2 != 1) : 1));
#pragma unroll
      for (int e = 0; e < CH; ++e) S[j1 * 3 + j2][e] = fmaf(x[e], wgt, S[j1 * 3 + j2][e]);
    }
  }
}

// Pass P of the window sums covers the lane's channel vectors P PV .. P PV +
// PV - 1 (W = PV VEC channels).  use = false: the loads still happen (at a
// valid address) but add nothing.
template <int R, int JD, int CIN, int PV, int P>
__device__ __forceinline__ void summary_add(float (&S)[9][PV * cell_vec<CIN>()],
                                            const float* __restrict__ p, bool use) {
  using K = CellCfg<CIN, 1>;
  constexpr int CH = PV * K::VEC;
  constexpr int dir0 = R / 9 - 1, dir1 = (R / 3) % 3 - 1, dir2 = R % 3 - 1;
#pragma unroll
  for (int ed = -1; ed <= 1; ++ed) {
    if (dir0 != 0 ? ed != -dir0 : (ed != 0 && ed != 1 - JD)) continue;
#pragma unroll
    for (int eh = -1; eh <= 1; ++eh) {
      if (dir1 != 0 && eh != -dir1) continue;
#pragma unroll
      for (int ew = -1; ew <= 1; ++ew) {
        if (dir2 != 0 && ew != -dir2) continue;
        float v[CH];
#pragma unroll
        for (int i = 0; i < PV; ++i) {
          const typename K::Vec q = *reinterpret_cast<const typename K::Vec*>(
              p + bset(ed, eh, ew) * CIN + K::VSTRIDE * (P * PV + i));
#pragma unroll
          for (int e = 0; e < K::VEC; ++e) v[K::VEC * i + e] = use ? vget<K::VEC>(q, e) : 0.f;
        }
        const bool n0 = dir0 == 0 && ed != 0;
#pragma unroll
        for (int j1 = 0; j1 < 3; ++j1) {
          if (dir1 != 0 ? j1 != dir1 + 1 : (eh != 0 && j1 != 1 - eh)) continue;
          const bool n1 = n0 != (dir1 == 0 && eh != 0);
#pragma unroll
          for (int j2 = 0; j2 < 3; ++j2) {
            if (dir2 != 0 ? j2 != dir2 + 1 : (ew != 0 && j2 != 1 - ew)) continue;
            const bool neg = n1 != (dir2 == 0 && ew != 0);
#pragma unroll
            for (int e = 0; e < CH; ++e) S[j1 * 3 + j2][e] += neg ? -v[e] : v[e];
          }
        }
      }
    }
  }
}

// TRIV: the cell's face and edge neighbour trees are known to be unsplit, so
// all its codes are rows, as corner codes always are; then the row gather is
// issued whatever the code (a code that is not a row reads zeros), so that
// it need not wait behind a branch.
// The lane's channel vectors P PV .. P PV + PV - 1 of row `row` (off: the
// byte offset of the lane's first channel).
template <int CIN, int PV, int P, class G>
__device__ __forceinline__ void gather_pass(const G& rin, uint32_t row, uint32_t off,
                                            float (&x)[PV * cell_vec<CIN>()]) {
  using K = CellCfg<CIN, 1>;
#pragma unroll
  for (int i = 0; i < PV; ++i) {
    const typename K::Vec v = gather_at<K::VEC>(rin, row, off + 4u * K::VSTRIDE * (P * PV + i));
#pragma unroll
    for (int e = 0; e < K::VEC; ++e) x[K::VEC * i + e] = vget<K::VEC>(v, e);
  }
}

template <int R, int JD, int SZ, int CIN, bool TRIV, int PV, int P, class G>
__device__ __forceinline__ void region_sum(float (&S)[9][PV * cell_vec<CIN>()], int32_t code, const G& rin,
                                           const float* __restrict__ bsum, int choff) {
  constexpr int CH = PV * cell_vec<CIN>();
  constexpr int nz = (R / 9 != 1) + ((R / 3) % 3 != 1) + (R % 3 != 1);
  if constexpr (TRIV || nz == 3) {  // codes are rows (or outside)
    float x[CH];
    gather_pass<CIN, PV, P>(rin, G::addr(code), 4u * choff, x);
    region_add<R, JD, SZ, CH>(S, x);
  } else if (code >= 0) {
    float x[CH];
    gather_pass<CIN, PV, P>(rin, G::addr(code), 4u * choff, x);
    region_add<R, JD, SZ, CH>(S, x);
  } else if (code <= -2) {
    summary_add<R, JD, CIN, PV, P>(S, bsum + (int64_t)(-2 - code) * (kSets * CIN) + choff, true);
  }
}

// The regions of layer JD (those with dir_d in {0, JD - 1}), R ascending:
// their codes are loaded first, then the regions are added a few at a time.
template <int JD>
constexpr bool in_layer(int R) {
  return R != 13 && (R / 9 - 1 == 0 || R / 9 - 1 == JD - 1);
}

template <int R, int JD, int SZ, int CIN, bool TRIV, int PV, int P>
struct RegionLayer {
  static constexpr int W = PV * cell_vec<CIN>();
  __device__ __forceinline__ static void codes(int32_t (&c)[27], const int32_t* __restrict__ col,
                                               int64_t ccap) {
    if constexpr (in_layer<JD>(R)) c[R] = col[(int64_t)(R - (R > 13)) * ccap];
    RegionLayer<R + 1, JD, SZ, CIN, TRIV, PV, P>::codes(c, col, ccap);
  }
  template <class G>
  __device__ __forceinline__ static void run(float (&S)[9][W], const int32_t (&c)[27], const G& rin,
                                             const float* bsum, int choff) {
    if constexpr (in_layer<JD>(R)) {
      region_sum<R, JD, SZ, CIN, TRIV, PV, P>(S, c[R], rin, bsum, choff);
      // A few regions' loads in flight at a time (more would spill).
      if constexpr (R % OC_REGION_GROUP == OC_REGION_GROUP - 1) __builtin_amdgcn_sched_barrier(0);
    }
    RegionLayer<R + 1, JD, SZ, CIN, TRIV, PV, P>::run(S, c, rin, bsum, choff);
  }
};
template <int JD, int SZ, int CIN, bool TRIV, int PV, int P>
struct RegionLayer<27, JD, SZ, CIN, TRIV, PV, P> {
  static constexpr int W = PV * cell_vec<CIN>();
  __device__ __forceinline__ static void codes(int32_t (&)[27], const int32_t*, int64_t) {}
  template <class G>
  __device__ __forceinline__ static void run(float (&)[9][W], const int32_t (&)[27], const G&, const float*,
                                             int) {}
};

// Batched form of a layer's regions (the default): the regions' loads are
// issued in groups and added once the whole group is in, instead of one
// region at a time behind a branch on its code.
//   - Rows: every region of the layer, the gather made whatever the code (a
//     code that is not a row reads zeros), RG regions per group.
//   - Boundary sums: regions that can be split (faces and edges), only when
//     some lane of the wave has that region split (a wave-uniform branch);
//     lanes whose region is a row read zeros.  Groups hold up to SB sets.
// A lane's region is either a row or split, so each adds exactly what the
// one-region form adds.
#ifndef OC_CELLR_BATCH
#define OC_CELLR_BATCH 1
#endif
#ifndef OC_CELLR_ROW_GROUP
#define OC_CELLR_ROW_GROUP 17
#endif
#ifndef OC_CELLR_SET_GROUP
#define OC_CELLR_SET_GROUP 18
#endif

struct RegionList {
  int n;
  int r[26];
};

constexpr int region_nz(int R) { return (R / 9 != 1) + ((R / 3) % 3 != 1) + (R % 3 != 1); }

// The regions of layer JD (all of them, or those that can be split).
constexpr RegionList layer_list(int JD, bool splittable) {
  RegionList l{0, {}};
  for (int R = 0; R < 27; ++R) {
    const int nz = region_nz(R);
    if (R == 13 || !(R / 9 - 1 == 0 || R / 9 - 1 == JD - 1)) continue;
    if (splittable && nz == 3) continue;  // corners are always one leaf
    l.r[l.n++] = R;
  }
  return l;
}

// Boundary sets that layer JD reads of split region R (as summary_add).
constexpr int layer_sets(int R, int JD) {
  const int d0 = R / 9 - 1, d1 = (R / 3) % 3 - 1, d2 = R % 3 - 1;
  return (d0 != 0 ? 1 : (JD == 1 ? 1 : 2)) * (d1 != 0 ? 1 : 3) * (d2 != 0 ? 1 : 3);
}

// End of the set group (at most SB sets) that starts at list entry k0.
constexpr int set_group_end(int JD, int k0, int SB) {
  const RegionList l = layer_list(JD, true);
  int k = k0, n = 0;
  while (k < l.n && (k == k0 || n + layer_sets(l.r[k], JD) <= SB)) n += layer_sets(l.r[k++], JD);
  return k;
}
constexpr int set_group_offset(int JD, int k0, int k) {
  int n = 0;
  for (int i = k0; i < k; ++i) n += layer_sets(layer_list(JD, true).r[i], JD);
  return n;
}

// Loads of the sets of split region R that layer JD reads, in summary_add's
// order, into y[O ..]; a = the slot's first set row (or no row), rs: the
// boundary sums as rows of CIN floats.
template <int R, int JD, int CIN, int PV, int P, int O, int NB, class G>
__device__ __forceinline__ void summary_load(float (&y)[NB][PV * cell_vec<CIN>()], const G& rs, uint32_t a,
                                             int choff) {
  using K = CellCfg<CIN, 1>;
  constexpr int dir0 = R / 9 - 1, dir1 = (R / 3) % 3 - 1, dir2 = R % 3 - 1;
  int j = O;
#pragma unroll
  for (int ed = -1; ed <= 1; ++ed) {
    if (dir0 != 0 ? ed != -dir0 : (ed != 0 && ed != 1 - JD)) continue;
#pragma unroll
    for (int eh = -1; eh <= 1; ++eh) {
      if (dir1 != 0 && eh != -dir1) continue;
#pragma unroll
      for (int ew = -1; ew <= 1; ++ew) {
        if (dir2 != 0 && ew != -dir2) continue;
#pragma unroll
        for (int i = 0; i < PV; ++i) {
          const typename K::Vec q = gather_at<K::VEC>(
              rs, a, 4u * (uint32_t)(bset(ed, eh, ew) * CIN + choff + K::VSTRIDE * (P * PV + i)));
#pragma unroll
          for (int e = 0; e < K::VEC; ++e) y[j][K::VEC * i + e] = vget<K::VEC>(q, e);
        }
        ++j;
      }
    }
  }
}

// summary_add over sets already loaded (y[O ..], the order of summary_load).
template <int R, int JD, int CIN, int PV, int O, int NB>
__device__ __forceinline__ void summary_add_loaded(float (&S)[9][PV * cell_vec<CIN>()],
                                                   const float (&y)[NB][PV * cell_vec<CIN>()]) {
  constexpr int CH = PV * cell_vec<CIN>();
  constexpr int dir0 = R / 9 - 1, dir1 = (R / 3) % 3 - 1, dir2 = R % 3 - 1;
  int j = O;
#pragma unroll
  for (int ed = -1; ed <= 1; ++ed) {
    if (dir0 != 0 ? ed != -dir0 : (ed != 0 && ed != 1 - JD)) continue;
#pragma unroll
    for (int eh = -1; eh <= 1; ++eh) {
      if (dir1 != 0 && eh != -dir1) continue;
#pragma unroll
      for (int ew = -1; ew <= 1; ++ew) {
        if (dir2 != 0 && ew != -dir2) continue;
        const bool n0 = dir0 == 0 && ed != 0;
#pragma unroll
        for (int j1 = 0; j1 < 3; ++j1) {
          if (dir1 != 0 ? j1 != dir1 + 1 : (eh != 0 && j1 != 1 - eh)) continue;
          const bool n1 = n0 != (dir1 == 0 && eh != 0);
#pragma unroll
          for (int j2 = 0; j2 < 3; ++j2) {
            if (dir2 != 0 ? j2 != dir2 + 1 : (ew != 0 && j2 != 1 - ew)) continue;
            const bool neg = n1 != (dir2 == 0 && ew != 0);
#pragma unroll
            for (int e = 0; e < CH; ++e) S[j1 * 3 + j2][e] += neg ? -y[j][e] : y[j][e];
          }
        }
        ++j;
      }
    }
  }
}

// Row groups: list entries [K, K1) (at most RG) loaded, then added; then the
// next group.
template <int JD, int K, int SZ, int CIN, int PV, int P, int RG = OC_CELLR_ROW_GROUP>
struct RowGroups {
  static constexpr int W = PV * cell_vec<CIN>();
  static constexpr int N = layer_list(JD, false).n;
  template <int I, int K1, class G>
  __device__ __forceinline__ static void load(float (&x)[RG][W], const int32_t (&c)[27],
                                              const G& rin, int choff) {
    if constexpr (I < K1) {
      constexpr int R = layer_list(JD, false).r[I];
      const int32_t code = c[R];
      gather_pass<CIN, PV, P>(rin, G::addr(code >= 0 ? code : -1), 4u * choff, x[I - K]);
      load<I + 1, K1>(x, c, rin, choff);
    }
  }
  template <int I, int K1>
  __device__ __forceinline__ static void add(float (&S)[9][W], const float (&x)[RG][W]) {
    if constexpr (I < K1) {
      constexpr int R = layer_list(JD, false).r[I];
      region_add<R, JD, SZ, W>(S, x[I - K]);
      add<I + 1, K1>(S, x);
    }
  }
  template <class G>
  __device__ __forceinline__ static void run(float (&S)[9][W], const int32_t (&c)[27], const G& rin, int choff) {
    if constexpr (K < N) {
      constexpr int K1 = K + RG < N ? K + RG : N;
      float x[RG][W];
      load<K, K1>(x, c, rin, choff);
      __builtin_amdgcn_sched_barrier(0);
      add<K, K1>(S, x);
      __builtin_amdgcn_sched_barrier(0);
      RowGroups<JD, K1, SZ, CIN, PV, P, RG>::run(S, c, rin, choff);
    }
  }
};

// Set groups of the splittable regions: list entries [K, K1) (at most SB
// sets, or one region) whose region some lane has split, loaded, then
// added; then the next group.
template <int JD, int K, int CIN, int PV, int P, int SB = OC_CELLR_SET_GROUP>
struct SetGroups {
  static constexpr int W = PV * cell_vec<CIN>();
  static constexpr int N = layer_list(JD, true).n;
  static constexpr int NB = SB > 9 ? SB : 9;
  template <int I, int K1, class G>
  __device__ __forceinline__ static void load(float (&y)[NB][W], const int32_t (&c)[27], uint32_t need,
                                              const G& rs, int choff) {
    if constexpr (I < K1) {
      constexpr int R = layer_list(JD, true).r[I];
      if (need & (1u << (I - K))) {
        const int32_t code = c[R];
        summary_load<R, JD, CIN, PV, P, set_group_offset(JD, K, I), NB>(
            y, rs, G::addr(code <= -2 ? kSets * (-2 - code) : -1), choff);
      }
      load<I + 1, K1>(y, c, need, rs, choff);
    }
  }
  template <int I, int K1>
  __device__ __forceinline__ static void add(float (&S)[9][W], const float (&y)[NB][W], uint32_t need) {
    if constexpr (I < K1) {
      constexpr int R = layer_list(JD, true).r[I];
      if (need & (1u << (I - K))) summary_add_loaded<R, JD, CIN, PV, set_group_offset(JD, K, I), NB>(S, y);
      add<I + 1, K1>(S, y, need);
    }
  }
  template <int I, int K1>
  __device__ __forceinline__ static uint32_t needed(const int32_t (&c)[27]) {
    if constexpr (I < K1) {
      constexpr int R = layer_list(JD, true).r[I];
      const uint32_t any = __ballot(c[R] <= -2) != 0ull ? 1u : 0u;
      return (any << (I - K)) | needed<I + 1, K1>(c);
    } else {
      return 0u;
    }
  }
  template <class G>
  __device__ __forceinline__ static void run(float (&S)[9][W], const int32_t (&c)[27], const G& rs, int choff) {
    if constexpr (K < N) {
      constexpr int K1 = set_group_end(JD, K, SB);
      const uint32_t need = __builtin_amdgcn_readfirstlane(needed<K, K1>(c));
      if (need != 0u) {
        float y[NB][W];
        load<K, K1>(y, c, need, rs, choff);
        __builtin_amdgcn_sched_barrier(0);
        add<K, K1>(S, y, need);
        __builtin_amdgcn_sched_barrier(0);
      }
      SetGroups<JD, K1, CIN, PV, P, SB>::run(S, c, rs, choff);
    }
  }
};

// Contract pass P (vectors P PV .. + PV - 1) of layer JD into acc.
template <int CIN, int NT, int JD, int PV, int P>
__device__ __forceinline__ void contract_pass(const float (&S)[9][PV * cell_vec<CIN>()],
                                              const float* wl, int lane,
                                              typename CellCfg<CIN, NT>::Acc (&acc)[NT]) {
  using K = CellCfg<CIN, NT>;
#pragma unroll
  for (int k = 0; k < 9; ++k) {
    const int dl = 9 * JD + k;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < PV; ++i) {
        const int jv = P * PV + i;
        const typename K::Vec bv =
            reinterpret_cast<const typename K::Vec*>(wl)[((dl * NT + nt) * K::NV + jv) * 64 + lane];
#pragma unroll
        for (int e = 0; e < K::VEC; ++e)
          acc[nt] = mfma<16>(S[k][K::VEC * i + e], vget<K::VEC>(bv, e), acc[nt]);
      }
    if (k % 3 == 2) __builtin_amdgcn_sched_barrier(0);  // bounds the B loads in flight
  }
}

// As contract_pass, for window sums held in the gather layout: the A
// operand of MFMA lane L comes from lane perm / 4.
template <int CIN, int NT, int JD, int PV, int P>
__device__ __forceinline__ void contract_pass_perm(const float (&S)[9][PV * cell_vec<CIN>()],
                                                   const float* wl, int lane, int perm,
                                                   typename CellCfg<CIN, NT>::Acc (&acc)[NT]) {
  using K = CellCfg<CIN, NT>;
  constexpr int W = PV * K::VEC;
#pragma unroll
  for (int k = 0; k < 9; ++k) {
    // One window sum at a time, so that few moved values are live.
    float T[W];
#pragma unroll
    for (int e = 0; e < W; ++e)
      T[e] = __builtin_bit_cast(float, __builtin_amdgcn_ds_bpermute(perm, __builtin_bit_cast(int, S[k][e])));
    const int dl = 9 * JD + k;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int i = 0; i < PV; ++i) {
        const int jv = P * PV + i;
        const typename K::Vec bv =
            reinterpret_cast<const typename K::Vec*>(wl)[((dl * NT + nt) * K::NV + jv) * 64 + lane];
#pragma unroll
        for (int e = 0; e < K::VEC; ++e)
          acc[nt] = mfma<16>(T[K::VEC * i + e], vget<K::VEC>(bv, e), acc[nt]);
      }
    if (k % 3 == 2) __builtin_amdgcn_sched_barrier(0);  // bounds the B loads in flight
  }
}

// Lane layout of the edge-4/8 kernels' window sums.  The MFMA layout (lane
// m + 16 g: channel chunk g of cell m) has the 16 lanes that the memory
// pipeline serves together read 16 rows; the gather layout (lane l: chunk
// l % 4 of cell 4 (l / 16) + (l / 4) % 4) has them read 4 rows, 64
// contiguous bytes each, and the sums move to the MFMA layout by
// ds_bpermute before each contraction.
#ifndef OC_CELLR_GATHER_LAYOUT
#define OC_CELLR_GATHER_LAYOUT 1
#endif
// The cell and channel chunk of a lane, and the ds_bpermute address that
// fetches the MFMA lane's operand.
__device__ __forceinline__ int cellr_cell(int lane) {
  return OC_CELLR_GATHER_LAYOUT ? 4 * (lane >> 4) + ((lane >> 2) & 3) : lane % 16;
}
__device__ __forceinline__ int cellr_chunk(int lane) { return OC_CELLR_GATHER_LAYOUT ? lane & 3 : lane / 16; }
__device__ __forceinline__ int cellr_perm(int lane) {
  return 4 * (16 * ((lane & 15) >> 2) + 4 * (lane & 3) + (lane >> 4));
}
// The lane that holds cell i (i < 16) in the kernels' layout.
__device__ __forceinline__ int cellr_lane(int i) {
  return OC_CELLR_GATHER_LAYOUT ? 16 * (i >> 2) + 4 * (i & 3) : i;
}

// One layer of the window sums, in NV / PV passes over the lane's channel
// vectors (fewer registers per pass; the codes are loaded once per layer).
template <int CIN, int NT, int SZ, bool TRIV, int JD, int PV, int P>
struct LayerPasses {
  template <class G, class GS>
  __device__ __forceinline__ static void run(const int32_t (&c)[27], const float (&xs)[CIN / 4],
                                             bool live, const G& rin, const GS& rs,
                                             const float* bsum, int choff, const float* wl,
                                             int lane, typename CellCfg<CIN, NT>::Acc (&acc)[NT]) {
    using K = CellCfg<CIN, NT>;
    constexpr int W = PV * K::VEC;
    if constexpr (P * PV < K::NV) {
      float xp[W];
#pragma unroll
      for (int e = 0; e < W; ++e) xp[e] = xs[P * W + e];
      float S[9][W];
      init_layer<SZ, JD>(S, xp);
      if constexpr (OC_CELLR_BATCH && !TRIV) {
        // c holds -1 (outside: nothing) for lanes without a cell.
        RowGroups<JD, 0, SZ, CIN, PV, P>::run(S, c, rin, choff);
        SetGroups<JD, 0, CIN, PV, P>::run(S, c, rs, choff);
      } else {
        if (live) RegionLayer<0, JD, SZ, CIN, TRIV, PV, P>::run(S, c, rin, bsum, choff);
      }
      if constexpr (OC_CELLR_GATHER_LAYOUT)
        contract_pass_perm<CIN, NT, JD, PV, P>(S, wl, lane, cellr_perm(lane), acc);
      else
        contract_pass<CIN, NT, JD, PV, P>(S, wl, lane, acc);
      __builtin_amdgcn_sched_barrier(0);
      LayerPasses<CIN, NT, SZ, TRIV, JD, PV, P + 1>::run(c, xs, live, rin, rs, bsum, choff, wl, lane,
                                                        acc);
    }
  }
};

#ifndef OC_CELLR_THREADS
#define OC_CELLR_THREADS 512
#endif
#ifndef OC_CELLR_PV
#define OC_CELLR_PV 1
#endif
constexpr int kCellrThreads = OC_CELLR_THREADS;

// GP gathers the input rows, GS the boundary sums (as rows of CIN floats).
template <int CIN, int NT, int SZ, bool TRIV, class GP, class GS>
__device__ __forceinline__ void cellr_tiles(
    const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix, int gd, int gh, int gw,
    int64_t n_leaves, const uint64_t* __restrict__ info, const int32_t* __restrict__ brow,
    const int64_t* __restrict__ meta, int kind, const int32_t* __restrict__ codes,
    const float* __restrict__ bsum, uint32_t n_sum_rows, int64_t ccap, const float* __restrict__ in,
    const float* __restrict__ wm, uint32_t n_rows, const float* __restrict__ bias, int cout,
    int relu, float* __restrict__ out, const int64_t* __restrict__ kpre, int64_t t0, int64_t t1) {
  // Channel blocks: blockIdx.y selects an output block (its weight layout
  // and its [n_leaves][cout] destination).
  wm += (int64_t)blockIdx.y * MfmaCfg<CIN, NT, 16>::WFLOATS;
  out += (int64_t)blockIdx.y * n_leaves * cout;
  if (bias != nullptr) bias += (int64_t)blockIdx.y * cout;
  using K = CellCfg<CIN, NT>;
  constexpr int CH = K::CH;
  // Channel vectors per window-sum pass.
  constexpr int PV = OC_CELLR_PV < K::NV ? OC_CELLR_PV : K::NV;
  extern __shared__ float smem[];
  float* wl = smem;
  weights_to_lds<CIN, NT, 16>(wm, wl);
  const GP rin = GP::make(in, n_rows);
  const GS rs = GS::make(bsum, n_sum_rows);  // the boundary sums, as rows of CIN floats
  const int lane = threadIdx.x & 63;
  int64_t lbeg, lcnt;
  kind_range(meta, kind, n_leaves, lbeg, lcnt);
  {
    // Only the cells of trees [t0, t1) (kpre: the kind's per-tree prefix).
    const int64_t a = min(lcnt, max((int64_t)0, kpre[t0]));
    const int64_t b = min(lcnt, max(a, kpre[t1]));
    lbeg += a;
    lcnt = b - a;
  }
  const WaveTiles wt = wave_tiles((lcnt + 15) / 16);
  const int m = cellr_cell(lane), g = cellr_chunk(lane);
  const int choff = K::VEC * g;  // the lane's first channel
  float bvals[NT];
  bias16<NT>(bias, cout, lane, bvals);
  for (int64_t tile = wt.first; tile < wt.end; tile += wt.stride) {
    const int64_t idx = tile * 16 + m;
    int row = idx < lcnt ? brow[lbeg + idx] : -1;
    if (row >= n_leaves || lbeg + idx >= ccap) row = -1;  // only a non-canonical structure
    const int32_t* col = codes + (lbeg + idx);  // the cell's column of region codes
    float xs[CH];
    gather_channels_at<CIN>(rin, GP::addr(row), 4u * choff, xs);
    typename K::Acc acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[nt][r] = 0.f;
#pragma unroll
    for (int jd = 0; jd < 3; ++jd) {
      int32_t c[27];
#pragma unroll
      for (int r = 0; r < 27; ++r) c[r] = -1;
      if (row >= 0) {
        if (jd == 0) RegionLayer<0, 0, SZ, CIN, TRIV, 1, 0>::codes(c, col, ccap);
        if (jd == 1) RegionLayer<0, 1, SZ, CIN, TRIV, 1, 0>::codes(c, col, ccap);
        if (jd == 2) RegionLayer<0, 2, SZ, CIN, TRIV, 1, 0>::codes(c, col, ccap);
      }
      if (jd == 0) LayerPasses<CIN, NT, SZ, TRIV, 0, PV, 0>::run(c, xs, row >= 0, rin, rs, bsum, choff, wl, lane, acc);
      if (jd == 1) LayerPasses<CIN, NT, SZ, TRIV, 1, PV, 0>::run(c, xs, row >= 0, rin, rs, bsum, choff, wl, lane, acc);
      if (jd == 2) LayerPasses<CIN, NT, SZ, TRIV, 2, PV, 0>::run(c, xs, row >= 0, rin, rs, bsum, choff, wl, lane, acc);
      __builtin_amdgcn_sched_barrier(0);  // keeps the next layer's loads out of this one
    }
    // The row of cell m, for the store's MFMA layout.
    const int row_m = OC_CELLR_GATHER_LAYOUT ? __builtin_amdgcn_ds_bpermute(cellr_perm(lane), row) : row;
    store_tile16<NT>(acc, row_m, (relu & 2) ? 1.f : 1.f / (float)(SZ * SZ * SZ), lane, bvals, cout, relu,
                     out);
  }
}

// The boundary sums are gathered through 32-bit offsets (RowsRaw) when the
// structure's slots (their count read on the device, *slot_total: a
// workspace sized by the bound may hold far more) span less than 4 GiB of
// sums and the input does too, else through 64-bit addresses.
template <int CIN, int NT, int SZ, bool TRIV, class GP>
__global__ void __launch_bounds__(kCellrThreads) k_conv_cellr_mfma(
    const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix, int gd, int gh, int gw,
    int64_t n_leaves, const uint64_t* __restrict__ info, const int32_t* __restrict__ brow,
    const int64_t* __restrict__ meta, int kind, const int32_t* __restrict__ codes,
    const float* __restrict__ bsum, const int64_t* __restrict__ slot_total, int64_t cap, int64_t ccap,
    const float* __restrict__ in, const float* __restrict__ wm, uint32_t n_rows,
    const float* __restrict__ bias, int cout, int relu, float* __restrict__ out,
    const int64_t* __restrict__ kpre, int64_t t0, int64_t t1) {
  int64_t ns = slot_total[0];
  ns = ns < 0 ? 0 : (ns > cap ? cap : ns);
  const bool raw = std::is_same<GP, RowsRaw<CIN>>::value &&
                   (uint64_t)ns * kSets * (uint64_t)CIN * 4u < (uint64_t)kOutside;
  if (raw)
    cellr_tiles<CIN, NT, SZ, TRIV, GP, RowsRaw<CIN>>(trees, prefix, gd, gh, gw, n_leaves, info, brow, meta, kind,
                                                     codes, bsum, (uint32_t)(ns * kSets), ccap, in, wm, n_rows,
                                                     bias, cout, relu, out, kpre, t0, t1);
  else
    cellr_tiles<CIN, NT, SZ, TRIV, GP, RowsWide<CIN>>(trees, prefix, gd, gh, gw, n_leaves, info, brow, meta, kind,
                                                      codes, bsum, 0u, ccap, in, wm, n_rows, bias, cout, relu, out,
                                                      kpre, t0, t1);
}

// Edge-8 cells whose face and edge neighbour trees are unsplit.  Every shell
// region is then one leaf's row (corners always are), so
// S_delta = sum_r w(delta, r) x_r over the cell's own row (r = 13) and its 26
// region rows, w(delta, r) being the number of region r's voxels in the
// window of delta, and Eq. 8 becomes out = b + sum_r W8_r x_r with effective
// weights W8_r = (1/512) sum_delta w(delta, r) W[1 - delta], formed once per
// weight set.  That is the unit voxels' gather-GEMM (K = 27 cin): MS cells
// per tile, term r's rows gathered into the A operand two terms ahead, the
// next tile's term rows loaded during this one.
template <int CIN, int NT, int MS, class GP>
__global__ void __launch_bounds__(kUnitThreads) k_conv_cell8t_gemm(
    int64_t n_leaves, const int32_t* __restrict__ brow, const int64_t* __restrict__ meta,
    const int32_t* __restrict__ codes, int64_t ccap, const float* __restrict__ in,
    const float* __restrict__ wm, uint32_t n_rows, const float* __restrict__ bias, int cout,
    int relu, float* __restrict__ out) {
  // Channel blocks: blockIdx.y selects an output block (its weight layout
  // and its [n_leaves][cout] destination).
  wm += (int64_t)blockIdx.y * MfmaCfg<CIN, NT, MS>::WFLOATS;
  out += (int64_t)blockIdx.y * n_leaves * cout;
  if (bias != nullptr) bias += (int64_t)blockIdx.y * cout;
  using C = MfmaCfg<CIN, NT, MS>;
  using Vec = typename VecT<C::VEC>::type;
  using Acc = typename AccT<MS>::type;
  const GP rin = GP::make(in, n_rows);
  extern __shared__ float smem[];
  float* wl = smem;
  weights_to_lds<CIN, NT, MS>(wm, wl);
  const int lane = threadIdx.x & 63;
  const int m = lane % MS, g = lane / MS, col = lane % MS;
  int64_t cnt = meta[0];  // the kind comes first in the lists
  if (cnt > ccap) cnt = ccap;
  if (cnt > n_leaves) cnt = n_leaves;
  const WaveTiles wt = wave_tiles((cnt + MS - 1) / MS);
  float bvals[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int co = MS * nt + col;
    bvals[nt] = (bias != nullptr && co < cout) ? bias[co] : 0.f;
  }
  // Term rows of the lane's cell in tile t (-1: none).
  int32_t trow[27];
  auto stage_load = [&](int64_t t) {
    const int64_t idx = t * MS + m;
    const bool ok = t < wt.end && idx < cnt;
#pragma unroll
    for (int r = 0; r < 27; ++r) {
      int32_t v = -1;
      if (ok) v = r == 13 ? brow[idx] : codes[(int64_t)(r - (r > 13)) * ccap + idx];
      trow[r] = v < n_leaves ? v : -1;  // only a non-canonical structure exceeds
    }
  };
  auto store_tile = [&](const Acc (&res)[NT], int srow) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int co = MS * nt + col;
#pragma unroll
      for (int r = 0; r < (MS == 32 ? 16 : 4); ++r) {
        const int i = MS == 32 ? 8 * (r / 4) + 4 * g + (r % 4) : 4 * g + r;
        const int rowi = __shfl(srow, i, 64);
        if (rowi < 0 || co >= cout) continue;
        float v = fmaf(res[nt][r], (relu & 2) ? 512.f : 1.f, bvals[nt]);
        if (relu & 1) v = fmaxf(v, 0.f);
        out[(int64_t)rowi * cout + co] = v;
      }
    }
  };
  constexpr int PD = unit_prefetch<CIN, MS>();
  static_assert(27 % (PD + 1) == 0, "the gather ring must line up across tiles");
  Vec abuf[PD + 1][C::NV];
  const uint32_t coff = 4u * C::VEC * g;  // the lane's first channel, in bytes
  auto gather_row = [&](uint32_t row, Vec* a) {
#pragma unroll
    for (int v = 0; v < C::NV; ++v) a[v] = gather_at<C::VEC>(rin, row, coff + 4 * C::VSTRIDE * v);
  };
  uint32_t aoff[27];
  auto offsets = [&]() {
#pragma unroll
    for (int r = 0; r < 27; ++r) aoff[r] = GP::addr(trow[r]);
  };
  Acc pacc[NT];
  int psrow = -1;
  bool have_prev = false;
  stage_load(wt.first);
  offsets();
#pragma unroll
  for (int k = 0; k < PD; ++k) gather_row(aoff[k], abuf[k]);
  for (int64_t tile = wt.first; tile < wt.end; tile += wt.stride) {
    const int srow = trow[13];
    Vec bbuf[2][NT][C::NV];
    auto load_b = [&](int dl, Vec (*b)[C::NV]) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const Vec* bsrc = reinterpret_cast<const Vec*>(wl) + ((dl * NT + nt) * C::NV) * 64 + lane;
#pragma unroll
        for (int v = 0; v < C::NV; ++v) b[nt][v] = bsrc[v * 64];
      }
    };
    Acc acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int r = 0; r < (MS == 32 ? 16 : 4); ++r) acc[nt][r] = 0.f;
    load_b(0, bbuf[0]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int dl = 0; dl < 27; ++dl) {
      if (dl + PD < 27) gather_row(aoff[dl + PD], abuf[(dl + PD) % (PD + 1)]);
      else gather_row(aoff[dl + PD - 27], abuf[(dl + PD) % (PD + 1)]);  // next tile
      if (dl + 1 < 27) load_b(dl + 1, bbuf[(dl + 1) % 2]);
      if (dl == 3) stage_load(tile + wt.stride);
      if (dl == 4 && have_prev) store_tile(pacc, psrow);
      if (dl == 22) {
        // The next tile's offsets (this tile's are no longer needed past
        // the gathers already issued).
#pragma unroll
        for (int k = 0; k < PD; ++k) aoff[k] = GP::addr(trow[k]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int v = 0; v < C::NV; ++v)
#pragma unroll
          for (int e = 0; e < C::VEC; ++e)
            acc[nt] = mfma<MS>(vget<C::VEC>(abuf[dl % (PD + 1)][v], e),
                               vget<C::VEC>(bbuf[dl % 2][nt][v], e), acc[nt]);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) pacc[nt] = acc[nt];
    psrow = srow;
    have_prev = true;
    offsets();  // the next tile's
  }
  if (have_prev) store_tile(pacc, psrow);
}

// Effective weights of the edge-8 gather-GEMM, in the unit kernel's B-operand
// order: term r (region dir = (r/9 - 1, (r/3)%3 - 1, r%3 - 1), r = 13 the cell
// itself) takes (1/sz^3) sum_delta w(delta, r) W[tap 1 - delta], where
// w(delta, r) = 0 unless delta_a = dir_a wherever dir_a != 0, and is the
// product of sz - |delta_a| over the other axes.
template <int CIN, int NT, int MS>
__global__ void k_eff_weights(const float* __restrict__ w, int cout, int sz,
                              float* __restrict__ wm) {
  using C = MfmaCfg<CIN, NT, MS>;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= C::WFLOATS) return;
  // Channel blocks: blockIdx.y selects a [cout][CIN][27] weight block.
  w += (int64_t)blockIdx.y * cout * CIN * 27;
  wm += (int64_t)blockIdx.y * C::WFLOATS;
  int q = idx;
  const int e = q % C::VEC; q /= C::VEC;
  const int lane = q % 64; q /= 64;
  const int jv = q % C::NV; q /= C::NV;
  const int nt = q % NT; q /= NT;
  const int r = q;
  const int co = MS * nt + lane % MS;
  const int ci = C::VEC * (C::KS * jv + lane / MS) + e;
  if (co >= cout) {
    wm[idx] = 0.f;
    return;
  }
  const int dir[3] = {r / 9 - 1, (r / 3) % 3 - 1, r % 3 - 1};
  double acc = 0.0;
  for (int dl = 0; dl < 27; ++dl) {
    const int dlt[3] = {dl / 9 - 1, (dl / 3) % 3 - 1, dl % 3 - 1};
    int wgt = 1;
    for (int a = 0; a < 3; ++a) {
      if (dir[a] != 0) wgt *= dlt[a] == dir[a] ? 1 : 0;
      else wgt *= sz - (dlt[a] != 0 ? 1 : 0);
    }
    if (wgt != 0) acc += (double)wgt * (double)w[((int64_t)co * CIN + ci) * 27 + (26 - dl)];
  }
  wm[idx] = (float)(acc / ((double)sz * sz * sz));
}

// Weights in B-operand order: for delta index dl, N-tile nt, vector jv, lane
// and element e: column co = MS*nt + lane%MS, channel ci = VEC*(KS*jv +
// lane/MS) + e, tap 26 - dl (Eq. 7 pairs input offset delta with tap 1 - delta).
template <int CIN, int NT, int MS>
__global__ void k_mfma_weights(const float* __restrict__ w, int cout, float* __restrict__ wm) {
  using C = MfmaCfg<CIN, NT, MS>;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= C::WFLOATS) return;
  // Channel blocks: blockIdx.y selects a [cout][CIN][27] weight block.
  w += (int64_t)blockIdx.y * cout * CIN * 27;
  wm += (int64_t)blockIdx.y * C::WFLOATS;
  int r = idx;
  const int e = r % C::VEC; r /= C::VEC;
  const int lane = r % 64; r /= 64;
  const int jv = r % C::NV; r /= C::NV;
  const int nt = r % NT; r /= NT;
  const int dl = r;
  const int co = MS * nt + lane % MS;
  const int ci = C::VEC * (C::KS * jv + lane / MS) + e;
  wm[idx] = co < cout ? w[((int64_t)co * CIN + ci) * 27 + (26 - dl)] : 0.f;
}

// ---------------------------------------------------------------------------
// Instantiated channel pairs.
// ---------------------------------------------------------------------------
typedef void (*MfmaFn)(int64_t, const int32_t*, const int64_t*, const float*, const float*,
                       uint32_t, const float*, int, int, float*);
typedef void (*CellFn)(const uint32_t*, const int64_t*, int, int, int, int64_t, const uint64_t*,
                       const int32_t*, const int64_t*, int, const int32_t*, const float*, const int64_t*,
                       int64_t, int64_t, const float*, const float*, uint32_t, const float*, int, int, float*,
                       const int64_t*, int64_t, int64_t);
typedef void (*WeightFn)(const float*, int, float*);
typedef void (*Cell8Fn)(int64_t, const int32_t*, const int64_t*, const int32_t*, int64_t,
                        const float*, const float*, uint32_t, const float*, int, int, float*);
typedef void (*Cell2Fn)(int64_t, const int32_t*, const int32_t*, const int32_t*, int64_t, const int64_t*,
                        const float*, const float*, uint32_t, const float*, int, int, float*);
typedef void (*EffWeightFn)(const float*, int, int, float*);
typedef void (*SumFn)(const uint32_t*, const int64_t*, const int32_t*, const int64_t*,
                      const int64_t*, int64_t, int64_t, const float*, uint32_t, float*,
                      const int64_t*, const int64_t*, int64_t, int64_t, const uint32_t*);

struct MfmaVariant {
  int cin, cout_max, cout_min, ms, nt;
  size_t wfloats;       // unit-voxel kernel weights (MS-row tiles)
  WeightFn weights;
  size_t cell_wfloats;  // cell kernels' weights (16-row tiles)
  WeightFn cell_weights;
  EffWeightFn eff_weights; // edge-8 effective weights (unit-kernel layout)
  // The kernels, [0] gathering through RowsRaw (input below 4 GiB), [1]
  // through RowsWide.
  MfmaFn kernel[2];
  Cell2Fn cell2[2];
  CellFn cell4[2], cell8[2];
  SumFn sums[2];
  Cell8Fn cell8g[2];    // edge-8 cells with unsplit face/edge neighbours
};

template <int CIN, int NT, int MS, int WIDE>
void set_kernels(MfmaVariant& v) {
  using C = MfmaCfg<CIN, NT, MS>;
  constexpr int CNT = (C::NCOL + 15) / 16;
  using G = typename std::conditional<WIDE != 0, RowsWide<CIN>, RowsRaw<CIN>>::type;
  v.kernel[WIDE] = &k_conv_unit_mfma<CIN, NT, MS, G>;
  v.cell2[WIDE] = &k_conv_cell2_mfma<CIN, CNT, G>;
  v.cell4[WIDE] = &k_conv_cellr_mfma<CIN, CNT, 4, false, G>;
  v.cell8[WIDE] = &k_conv_cellr_mfma<CIN, CNT, 8, false, G>;
  v.sums[WIDE] = &k_boundary_sums<CIN, G>;
  v.cell8g[WIDE] = &k_conv_cell8t_gemm<CIN, NT, MS, G>;
}

template <int CIN, int NT, int MS>
MfmaVariant make_variant(int cout_min) {
  using C = MfmaCfg<CIN, NT, MS>;
  MfmaVariant v;
  v.cin = CIN;
  v.cout_max = C::NCOL;
  v.cout_min = cout_min;
  v.ms = MS;
  v.nt = NT;
  v.wfloats = C::WFLOATS;
  v.weights = &k_mfma_weights<CIN, NT, MS>;
  constexpr int CNT = (C::NCOL + 15) / 16;
  v.cell_wfloats = MfmaCfg<CIN, CNT, 16>::WFLOATS;
  v.cell_weights = &k_mfma_weights<CIN, CNT, 16>;
  v.eff_weights = &k_eff_weights<CIN, NT, MS>;
  set_kernels<CIN, NT, MS, 0>(v);
  set_kernels<CIN, NT, MS, 1>(v);
  return v;
}

// cout in [cout_min, cout_max]; 32-wide tiles for cout 17..32, 16-wide ones
// for cout 1..16 (a tile column past cout holds zero weights and is not
// stored).
#ifndef OC_NARROW_COUT_MIN
#define OC_NARROW_COUT_MIN 1
#endif
const MfmaVariant* find_variant(int cin, int cout) {
  static const MfmaVariant table[] = {
#ifdef OC_UNIT_MS16
      make_variant<32, 2, 16>(17), make_variant<16, 2, 16>(17), make_variant<8, 2, 16>(17),
      make_variant<4, 2, 16>(17),
#else
      make_variant<32, 1, 32>(17), make_variant<16, 1, 32>(17), make_variant<8, 1, 32>(17),
      make_variant<4, 1, 32>(17),
#endif
      make_variant<32, 1, 16>(OC_NARROW_COUT_MIN),  make_variant<16, 1, 16>(OC_NARROW_COUT_MIN),
      make_variant<8, 1, 16>(OC_NARROW_COUT_MIN),   make_variant<4, 1, 16>(OC_NARROW_COUT_MIN),
  };
  for (const MfmaVariant& v : table)
    if (v.cin == cin && cout >= v.cout_min && cout <= v.cout_max) return &v;
  return nullptr;
}

// Channel blocks for layers without a fused variant: cin a multiple of 32 and
// cout a multiple of 32 up to 256 (or below 32 with a variant of its own).
// Eq. 7 sums over input channels, so the layer is the sum over j of the
// convolutions of input channels [32j, 32j + 32) with the matching weight
// columns: it runs as J x K fused 32 -> cb convolutions; those of input
// block j write partial outputs [K][n_leaves][cb], which one kernel adds to
// the output (after the bias, before the ReLU) in block order.
struct Blocks {
  const MfmaVariant* v;  // the 32 -> cb variant; null when not blocked
  int J, K, cb;
};

Blocks conv_blocks(int cin, int cout) {
  Blocks b{nullptr, 0, 0, 0};
  if (find_variant(cin, cout) != nullptr || cin % 32 != 0 || cin > 256 || cout > 256) return b;
  const int cb = cout % 32 == 0 ? 32 : cout;
  if (cb != 32 && cout > 32) return b;
  b.v = find_variant(32, cb);
  if (b.v == nullptr) return b;
  b.J = cin / 32;
  b.K = cout / cb;
  b.cb = cb;
  return b;
}

// Weight blocks: wb[(j K + k)][co][ci][t] = w[cb k + co][32 j + ci][t].
__global__ void k_weight_blocks(const float* __restrict__ w, int cin, int cout, int cb,
                                float* __restrict__ wb) {
  const int64_t n = 27LL * cin * cout;
  const int K = cout / cb;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    int64_t r = i;
    const int t = (int)(r % 27); r /= 27;
    const int ci = (int)(r % 32); r /= 32;
    const int co = (int)(r % cb); r /= cb;
    const int k = (int)(r % K);
    const int j = (int)(r / K);
    wb[i] = w[((int64_t)(cb * k + co) * cin + 32 * j + ci) * 27 + t];
  }
}

// xb[row][0..32) = x[row][32 j .. 32 j + 32): one float4 per thread (x and
// xb 16-byte aligned, cin a multiple of 32).
__global__ void k_channel_block(const float* __restrict__ x, int cin, int j, int64_t n_rows,
                                float* __restrict__ xb) {
  const int64_t n = n_rows * 8;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i >> 3;
    const int q = (int)(i & 7);
    reinterpret_cast<float4*>(xb)[i] = reinterpret_cast<const float4*>(x + row * cin + 32 * j)[q];
  }
}

// One input block's share of the output: out[row][cb k + c] = (first ? bias
// : out[row][cb k + c]) + part[k][row][c], then max(0, .) after the last
// block when relu is set.  Called for j = 0 .. J - 1 in order, it leaves
// act(bias + P_0 + P_1 + ...) summed in block order.
__global__ void k_block_accum(const float* __restrict__ part, int K, int cb, int64_t n_rows,
                              const float* __restrict__ bias, int first, int last, int relu,
                              float* __restrict__ out) {
  const int cout = K * cb;
  const int64_t n = n_rows * cout;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i / cout;
    const int co = (int)(i - row * cout);
    const int k = co / cb, c = co - k * cb;
    float v = first ? (bias ? bias[co] : 0.f) : out[i];
    v += part[((int64_t)k * n_rows + row) * cb + c];
    out[i] = (last && relu) ? fmaxf(v, 0.f) : v;
  }
}


// Chunks of trees for the boundary sums and the cells that read them (one:
// more chunks keep the sums in cache for their readers, but each chunk's
// launches then hold too few tiles per wave to hide their latency).
#ifndef OC_SUM_CHUNKS
#define OC_SUM_CHUNKS 1
#endif
constexpr int kSumChunks = OC_SUM_CHUNKS;

size_t mfma_smem(const MfmaVariant& v) {
  return sizeof(float) * v.wfloats + sizeof(int32_t) * (kUnitThreads / 64) * 2 * (v.ms / 8) * 64;
}

// Compute units and LDS bytes per workgroup of the current device, queried
// once per device (std::call_once: calls from several threads are safe).
struct DevLimits {
  int num_cus = 0;
  size_t max_smem = 0;
};

constexpr int kMaxDevices = 64;

struct DevSlot {
  std::once_flag once;
  hipError_t err = hipSuccess;
  DevLimits lim;
};

DevSlot g_devices[kMaxDevices];

hipError_t device_limits(DevLimits* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  DevSlot& d = g_devices[dev];
  std::call_once(d.once, [&d, dev]() {
    int cus = 0, smem = 0;
    hipError_t r = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (r == hipSuccess) r = hipDeviceGetAttribute(&smem, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    d.err = r;
    d.lim.num_cus = cus;
    d.lim.max_smem = (size_t)smem;
  });
  if (d.err != hipSuccess) return d.err;
  *out = d.lim;
  return hipSuccess;
}

// LDS bytes per workgroup for the support queries: the device's, or gfx950's
// 160 KB where none can be asked.
size_t smem_limit() {
  DevLimits L;
  return device_limits(&L) == hipSuccess ? L.max_smem : 160 * 1024;
}

// Workspace layout (each part 256-byte aligned):
//   leaf_info  u64 [n_leaves]                written by execute, for the generic and GEMM paths
//   wt         f32 [27 cin cout]            generic-kernel weights
//   wm         f32 [variant wfloats]        unit-voxel kernel B operands (if a variant exists)
//   wc         f32 [variant cell_wfloats]   cell kernels' B operands
//   w8         f32 [variant wfloats]        edge-8 effective weights (unit layout)
//   6 x (scan workspace (n_trees), i64 [n_trees + 1])
//              per tree: unit groups, each kind of larger cell, boundary-sum
//              slots -> prefixes
//   gkey       i64 [n_leaves / 8 + 1]
//   brow       i32 [n_leaves]
//   stl        i32 [n_trees]                split trees
//   meta       i64 [kKinds + 1]
//   nbt        i32 [(n_leaves / 8 + 1) 64]  unit-group neighbourhood rows (if a variant exists)
//   e2key      i32 [n_leaves]               edge-2 cells: node << 3 | octant (if a variant exists)
//   codes      i32 [26][ccap]               region codes of edge-4/8 cells (if a variant exists)
//   bkey       i64 [ccap]                   tree << 10 | bit of the edge-8/4 cells (if a variant exists)
//   sgemm, wblk, xblk, part                 GEMM window sums, channel blocks
// and last, the parts sized by the slot capacity cap (if a variant exists):
//   bsum       f32 [cap][26][cin]           boundary sums
//   ntab       i32 [cap][216]               6^3 rows around each split depth-1 node
//   smask      u32 [cap]                    boundary sets read per slot
// A slot belongs to a split tree or a split depth-1 node (a node table to
// the latter).  Every split node adds 7 leaves, so (n_leaves - n_trees) / 7
// slots hold every canonical structure of that size: the bound the size-only
// workspace query assumes.  A structure needs only its own count (split
// trees plus split depth-1 nodes, at least 1), which the exact query counts
// on the device; the capacity a call works with is what its workspace holds
// past the fixed parts (at most the bound).  A tree holds at most 8 cells of
// edge 4 or 8, so ccap = min(8 n_trees, n_leaves).
constexpr int kScans = 3 + kKinds;  // groups, the kinds, slots, split depth-1 nodes
constexpr int kSlotScan = 1 + kKinds;
constexpr int kNodeScan = 2 + kKinds;

struct ConvWs {
  uint64_t* info;
  float* wt;
  float* wm;
  float* wc;
  float* w8;
  char* scan[kScans];
  int64_t* pre[kScans];
  int64_t* gkey;
  int32_t* brow;
  int32_t* stl;
  int64_t* meta;
  float* bsum;
  int64_t cap;
  int32_t* nbt;
  int32_t* ntab;   // 6^3 tables of the split depth-1 nodes
  int64_t ncap;
  int32_t* e2key;  // per edge-2 cell: node << 3 | octant
  int64_t e2cap;
  int32_t* codes;
  int64_t ccap;
  int64_t* bkey;   // per edge-8/4 cell entry: tree << 10 | bit index
  uint32_t* smask;
  float* sgemm;  // window sums of one row chunk (GEMM path)
  float* wblk;   // channel blocks: weight blocks, one input block, partial outputs
  float* xblk;
  float* part;
  size_t total;
};

// Slot bound of a structure size (see the layout above).
int64_t slot_bound(int64_t n_trees, int64_t n_leaves) {
  return n_leaves > n_trees + 7 ? (n_leaves - n_trees) / 7 : 1;
}

// Bytes per slot of the slot-sized parts (each part's alignment aside).
size_t slot_bytes(int kcin) {
  return sizeof(float) * kSets * (size_t)kcin + sizeof(int32_t) * kNodeEntries + sizeof(uint32_t);
}

// slot_cap < 0: the bound.
ConvWs carve(void* base, int64_t n_trees, int64_t n_leaves, int cin, int cout, int64_t slot_cap = -1) {
  using oci::align256;
  char* p = static_cast<char*>(base);
  size_t off = 0;
  ConvWs w;
  auto take = [&](size_t bytes) {
    char* q = p ? p + off : nullptr;
    off += align256(bytes);
    return q;
  };
  // The fused kernels' variant: the layer's own, or the 32 -> cb one of its
  // channel blocks (one weight layout per block, 32-channel boundary sums).
  const Blocks bl = conv_blocks(cin, cout);
  const MfmaVariant* v = find_variant(cin, cout);
  const size_t nwl = v ? 1 : (bl.v ? (size_t)bl.J * bl.K : 0);
  const int kcin = v ? cin : 32;
  if (!v) v = bl.v;
  w.info = reinterpret_cast<uint64_t*>(take(sizeof(uint64_t) * (size_t)n_leaves));
  w.wt = reinterpret_cast<float*>(take(sizeof(float) * 27 * (size_t)cin * cout));
  w.wm = reinterpret_cast<float*>(take(v ? sizeof(float) * v->wfloats * nwl : 0));
  w.wc = reinterpret_cast<float*>(take(v ? sizeof(float) * v->cell_wfloats * nwl : 0));
  w.w8 = reinterpret_cast<float*>(take(v ? sizeof(float) * v->wfloats * nwl : 0));
  for (int k = 0; k < kScans; ++k) {
    w.scan[k] = take(oci::scan_workspace(n_trees));
    w.pre[k] = reinterpret_cast<int64_t*>(take(sizeof(int64_t) * (size_t)(n_trees + 1)));
  }
  w.gkey = reinterpret_cast<int64_t*>(take(sizeof(int64_t) * (size_t)(n_leaves / 8 + 1)));
  w.brow = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)n_leaves));
  w.stl = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)n_trees));
  w.meta = reinterpret_cast<int64_t*>(take(sizeof(int64_t) * (1 + kKinds)));
  // Also without a variant: the GEMM path gathers unit voxels' window sums
  // through it.
  w.nbt = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * 64 * (size_t)(n_leaves / 8 + 1)));
  w.e2cap = v ? n_leaves : 0;
  w.e2key = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (size_t)w.e2cap));
  w.ccap = v ? (8 * n_trees < n_leaves ? 8 * n_trees : n_leaves) : 0;
  w.codes = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * kSets * (size_t)w.ccap));
  w.bkey = reinterpret_cast<int64_t*>(take(sizeof(int64_t) * (size_t)w.ccap));
  w.sgemm = reinterpret_cast<float*>(take(oci::conv_gemm_buffer(n_leaves, cin)));
  w.wblk = reinterpret_cast<float*>(take(bl.v ? sizeof(float) * 27 * (size_t)cin * cout : 0));
  w.xblk = reinterpret_cast<float*>(take(bl.v ? sizeof(float) * 32 * (size_t)n_leaves : 0));
  w.part = reinterpret_cast<float*>(take(bl.v ? sizeof(float) * (size_t)n_leaves * cout : 0));
  // The slot-sized parts.  At least one slot where a variant exists: the
  // cell kernels may read slot 0 (and discard it) when no cell of a wave
  // needs boundary sums.
  const int64_t bound = slot_bound(n_trees, n_leaves);
  w.cap = v ? (slot_cap < 1 ? bound : (slot_cap < bound ? slot_cap : bound)) : 0;
  w.bsum = reinterpret_cast<float*>(take(sizeof(float) * kSets * (size_t)kcin * (size_t)w.cap));
  w.ncap = w.cap;
  w.ntab = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * kNodeEntries * (size_t)w.ncap));
  w.smask = reinterpret_cast<uint32_t*>(take(sizeof(uint32_t) * (size_t)w.cap));
  w.total = off + 256;
  return w;
}

// The slot capacity a workspace of ws_bytes holds (the bound at most), 0
// where no variant exists; -1 if it holds less than one slot.
int64_t slot_capacity(int64_t n_trees, int64_t n_leaves, int cin, int cout, size_t ws_bytes) {
  const ConvWs one = carve(nullptr, n_trees, n_leaves, cin, cout, 1);
  if (one.cap == 0) return ws_bytes >= one.total ? 0 : -1;
  if (ws_bytes < one.total) return -1;
  const int kcin = find_variant(cin, cout) ? cin : 32;
  // Each added slot adds slot_bytes over the three parts, whose alignment
  // padding may shrink by up to 3 x 255 bytes: start from that upper
  // estimate and step down to the largest capacity that fits.
  const size_t spare = ws_bytes - one.total;
  int64_t cap = 1 + (int64_t)((spare + 3 * 255) / slot_bytes(kcin));
  const int64_t bound = slot_bound(n_trees, n_leaves);
  if (cap > bound) cap = bound;
  while (cap > 1 && carve(nullptr, n_trees, n_leaves, cin, cout, cap).total > ws_bytes) --cap;
  return cap;
}

// Split trees plus split depth-1 nodes, added into *count (grid-stride, one
// atomic per workgroup).
__global__ void k_count_slots(const uint32_t* __restrict__ trees, int64_t n_trees,
                              unsigned long long* __restrict__ count) {
  __shared__ unsigned long long part[4];
  unsigned long long k = 0;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n_trees;
       t += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t w0 = trees[4 * t];
    if (w0 & 1u) k += 1 + __popc((w0 >> 1) & 0xFFu);
  }
  for (int o = 32; o > 0; o >>= 1) k += __shfl_xor(k, o, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = k;
  __syncthreads();
  if (threadIdx.x == 0) atomicAdd(count, part[0] + part[1] + part[2] + part[3]);
}

__global__ void k_zero_u64(unsigned long long* p) { *p = 0ull; }

// Output side of one fused pass: weight layouts, bias, width, epilogue mode
// and the [n_leaves][cout] destination.  relu: bit 0 applies max(0, .),
// bit 1 writes each cell's sum over its voxels instead of their mean (the
// bias still added once).
struct FusedOut {
  const float* wm;
  const float* wc;
  const float* w8;
  const float* bias;
  int cout, relu;
  float* out;
};

constexpr int kMaxOutBlocks = 8;
#ifndef OC_BLOCKED_MIN_LEAVES
#define OC_BLOCKED_MIN_LEAVES 65536
#endif
constexpr int64_t kBlockedMinLeaves = OC_BLOCKED_MIN_LEAVES;

// The fused kernels of variant v on input `in` (v->cin channels, n_rows
// rows) for nk output blocks (grid rows; block k's weight layouts and
// destination follow block k - 1's, as the kernels expect): unit voxels,
// edge-8 cells with unsplit neighbours and edge-2 cells, then the boundary
// sums of split nodes (once, they depend on the input only) and the edge-8
// and edge-4 cells that read them.
hipError_t fused_pass(const oci::ConvArgs& a, const ConvWs& w, const MfmaVariant* v, const float* in,
                      uint32_t n_rows, const FusedOut& o, int nk, const DevLimits& L, hipStream_t s) {
  const int num_cus = L.num_cus;
  const size_t max_smem = L.max_smem;
  // Raw buffer gathers below 4 GiB of input, 64-bit ones from there (the
  // edge-4/8 kernels pick their boundary sums' policy on the device).
  const int wide = (uint64_t)n_rows * (uint64_t)v->cin * 4u >= (uint64_t)kOutside ? 1 : 0;
  const size_t wsmem = sizeof(float) * v->cell_wfloats;
  const size_t msmem = mfma_smem(*v);
  if (msmem > max_smem) return hipErrorInvalidConfiguration;
  const int nblk = ((num_cus + 7) / 8) * 8;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(v->kernel[wide]),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)msmem);
  if (e != hipSuccess) return e;
  // Edge-8 cells with unsplit face and edge neighbours: the gather-GEMM with
  // effective weights (same LDS footprint as the unit kernel, no tables).
  const size_t gsm = sizeof(float) * v->wfloats;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(v->cell8g[wide]),
                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)gsm);
  if (e != hipSuccess) return e;
  auto launch_cells = [&](int k, int64_t t0, int64_t t1) -> hipError_t {
    const size_t smem = wsmem;
    if (smem > max_smem) return hipErrorInvalidConfiguration;
    const CellFn f = k == 1 || k == 0 ? v->cell8[wide] : v->cell4[wide];
    hipError_t r = hipFuncSetAttribute(reinterpret_cast<const void*>(f),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (r != hipSuccess) return r;
    hipLaunchKernelGGL(f, dim3(nblk, nk), dim3(kCellrThreads), smem, s, a.trees,
                       a.prefix, a.gd, a.gh, a.gw, a.n_leaves, (const uint64_t*)w.info,
                       (const int32_t*)w.brow, (const int64_t*)w.meta, k, (const int32_t*)w.codes,
                       (const float*)w.bsum, (const int64_t*)w.pre[kSlotScan] + a.n_trees, w.cap, w.ccap, in,
                       o.wc, n_rows, o.bias, o.cout, o.relu, o.out,
                       (const int64_t*)w.pre[1 + k], t0, t1);
    return hipGetLastError();
  };
  hipLaunchKernelGGL(v->kernel[wide], dim3(nblk, nk), dim3(kUnitThreads), msmem, s, a.n_leaves,
                     (const int32_t*)w.nbt, (const int64_t*)(w.pre[0] + a.n_trees), in, o.wm, n_rows,
                     o.bias, o.cout, o.relu, o.out);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(v->cell8g[wide], dim3(nblk, nk), dim3(kUnitThreads), gsm, s, a.n_leaves,
                     (const int32_t*)w.brow, (const int64_t*)w.meta, (const int32_t*)w.codes, w.ccap, in,
                     o.w8, n_rows, o.bias, o.cout, o.relu, o.out);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // Edge-2 cells (no boundary sums); the kernel keeps the shell offsets of
  // each wave's tile in LDS.
  {
    const size_t smem = wsmem + (size_t)(kMfmaThreads / 64) * kShell2Lds;
    if (smem > max_smem) return hipErrorInvalidConfiguration;
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(v->cell2[wide]),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(v->cell2[wide], dim3(nblk, nk), dim3(kMfmaThreads), smem, s, a.n_leaves,
                       (const int32_t*)w.brow, (const int32_t*)w.e2key, (const int32_t*)w.ntab, w.ncap,
                       (const int64_t*)w.meta, in, o.wc, n_rows, o.bias, o.cout, o.relu, o.out);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // Boundary sums and the cells that read them (other edge-8, edge-4), in
  // chunks of trees: the sums of the trees up to a chunk's end plus one tree
  // plane (every neighbour of its cells), then the chunk's cells, so that the
  // sums they read were written moments before and are still cached.
  const int64_t plane = (int64_t)a.gh * a.gw + a.gw + 1;
  const int64_t per_block = 4 * sum_trees_per_wave(v->cin);  // trees per pass of a 256-thread block
  int64_t done = 0;
  for (int c = 0; c < kSumChunks; ++c) {
    const int64_t t0 = a.n_trees * c / kSumChunks, t1 = a.n_trees * (c + 1) / kSumChunks;
    const int64_t need = c + 1 == kSumChunks ? a.n_trees : min(a.n_trees, t1 + plane);
    if (need > done) {
      int64_t blocks = (need - done + per_block - 1) / per_block;
      if (blocks > 8LL * num_cus) blocks = 8LL * num_cus;
      hipLaunchKernelGGL(v->sums[wide], dim3((unsigned)blocks), dim3(256), 0, s, a.trees, a.prefix,
                         (const int32_t*)w.stl, (const int64_t*)w.meta,
                         (const int64_t*)w.pre[kSlotScan], a.n_trees, w.cap, in, n_rows, w.bsum,
                         (const int64_t*)w.pre[1], (const int64_t*)w.pre[2], done, need,
                         (const uint32_t*)w.smask);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      done = need;
    }
    if (t1 > t0) {
      e = launch_cells(1, t0, t1);
      if (e != hipSuccess) return e;
      e = launch_cells(2, t0, t1);
      if (e != hipSuccess) return e;
    }
  }
  return hipGetLastError();
}

}  // namespace

namespace oci {

size_t conv_workspace(int64_t n_trees, int64_t n_leaves, int cin, int cout) {
  return carve(nullptr, n_trees, n_leaves, cin, cout).total;
}

size_t conv_workspace_slots(int64_t n_trees, int64_t n_leaves, int cin, int cout, int64_t slots) {
  return carve(nullptr, n_trees, n_leaves, cin, cout, slots < 1 ? 1 : slots).total;
}

int64_t conv_slot_capacity(int64_t n_trees, int64_t n_leaves, int cin, int cout, size_t ws_bytes) {
  return slot_capacity(n_trees, n_leaves, cin, cout, ws_bytes);
}

hipError_t launch_count_slots(const uint32_t* trees, int64_t n_trees, unsigned long long* count,
                              hipStream_t s) {
  hipLaunchKernelGGL(k_zero_u64, dim3(1), dim3(1), 0, s, count);
  int64_t blocks = (n_trees + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(k_count_slots, dim3((unsigned)blocks), dim3(256), 0, s, trees, n_trees, count);
  return hipGetLastError();
}

bool conv_mfma_supported(int cin, int cout) {
  const MfmaVariant* v = find_variant(cin, cout);
  if (!v) v = conv_blocks(cin, cout).v;
  if (!v) return false;
  // LDS: the whole weight set plus the neighbourhood rows of every wave must
  // fit one workgroup (160 KB on gfx950; the device is asked when present).
  return mfma_smem(*v) <= smem_limit();
}

int conv_auto_impl(int64_t n_leaves, int cin, int cout) {
  if (!conv_mfma_supported(cin, cout)) return 3;
  if (find_variant(cin, cout) != nullptr) return 2;
  // Channel blocks pay Cin/32 passes of six launches each, while the
  // window-sum GEMM writes and re-reads 27 Cin floats per leaf: the GEMM is
  // faster on small structures unless the input is wide (measured on
  // 32768 leaves: 64->64 and 64->128 favour the GEMM, 128->64 and 256->128
  // the blocks; on 4096 leaves the GEMM throughout).
  if (n_leaves >= kBlockedMinLeaves) return 2;
  return cin >= 128 && n_leaves >= kBlockedMinLeaves / 4 ? 2 : 3;
}

hipError_t launch_conv_prepare(const ConvArgs& a, void* ws, hipStream_t s) {
  const ConvWs w = carve(ws, a.n_trees, a.n_leaves, a.cin, a.cout, a.slot_cap);
  hipError_t e = hipSuccess;
  const int64_t nw = 27LL * a.cin * a.cout;
  hipLaunchKernelGGL(k_transpose_weights, dim3((unsigned)((nw + 255) / 256)), dim3(256), 0, s,
                     a.weight, a.cin, a.cout, w.wt);
  const MfmaVariant* v = find_variant(a.cin, a.cout);
  const Blocks bl = conv_blocks(a.cin, a.cout);
  if (v != nullptr || bl.v != nullptr) {
    // Channel blocks: the layouts of every weight block, one grid row each.
    const float* wsrc = a.weight;
    int wcout = a.cout;
    unsigned nb = 1;
    if (v == nullptr) {
      v = bl.v;
      hipLaunchKernelGGL(k_weight_blocks, dim3((unsigned)((nw + 255) / 256)), dim3(256), 0, s, a.weight,
                         a.cin, a.cout, bl.cb, w.wblk);
      wsrc = w.wblk;
      wcout = bl.cb;
      nb = (unsigned)(bl.J * bl.K);
    }
    hipLaunchKernelGGL(v->weights, dim3((unsigned)((v->wfloats + 255) / 256), nb), dim3(256), 0, s,
                       wsrc, wcout, w.wm);
    hipLaunchKernelGGL(v->cell_weights, dim3((unsigned)((v->cell_wfloats + 255) / 256), nb), dim3(256), 0,
                       s, wsrc, wcout, w.wc);
    hipLaunchKernelGGL(v->eff_weights, dim3((unsigned)((v->wfloats + 255) / 256), nb), dim3(256), 0, s,
                       wsrc, wcout, 8, w.w8);
  }
  const unsigned tb = (unsigned)((a.n_trees + 255) / 256);
  hipLaunchKernelGGL(k_leaf_kinds, dim3(tb), dim3(256), 0, s, a.trees, a.n_trees, a.gd, a.gh, a.gw,
                     scan_counts_buffer(w.scan[0]), scan_counts_buffer(w.scan[1]),
                     scan_counts_buffer(w.scan[2]), scan_counts_buffer(w.scan[3]),
                     scan_counts_buffer(w.scan[4]), scan_counts_buffer(w.scan[kSlotScan]),
                     scan_counts_buffer(w.scan[kNodeScan]));
  {
    void* sws[kScans];
    int64_t* spre[kScans];
    for (int k = 0; k < kScans; ++k) {
      sws[k] = w.scan[k];
      spre[k] = w.pre[k];
    }
    e = scan_counts_set(kScans, sws, a.n_trees, spre, s);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_leaf_lists, dim3(tb), dim3(256), 0, s, a.trees, a.prefix, w.pre[0], w.pre[1],
                     w.pre[2], w.pre[3], w.pre[4], (const int64_t*)w.pre[kNodeScan], a.n_trees, w.gkey,
                     w.brow, a.n_leaves / 8 + 1, a.n_leaves, w.stl, w.meta, w.e2key, w.e2cap, w.bkey,
                     w.ccap);
  if (w.cap > 0)
    hipLaunchKernelGGL(k_zero_u32, dim3((unsigned)((w.cap + 255) / 256)), dim3(256), 0, s, w.smask,
                       w.cap);
  DevLimits L;
  e = device_limits(&L);
  if (e != hipSuccess) return e;
  // Neighbourhood tables of the unit-voxel groups and the split depth-1 nodes.
  {
    // Up to a wave per split tree (their count is on the device), at most
    // OC_TREE_TABLE_BLOCKS workgroups per CU (the waves then take several
    // trees each instead of most of them exiting at once).
    int64_t blocks = (a.n_trees + kTreeWaves - 1) / kTreeWaves;
    const int64_t most = (int64_t)OC_TREE_TABLE_BLOCKS * L.num_cus;
    if (OC_TREE_TABLE_BLOCKS > 0 && blocks > most) blocks = most;
    if (blocks > (1LL << 30)) blocks = 1LL << 30;
    hipLaunchKernelGGL(k_tree_tables, dim3((unsigned)blocks), dim3(64 * kTreeWaves), 0, s, a.trees, a.prefix,
                       a.gd, a.gh, a.gw, a.n_trees, a.n_leaves, (const int32_t*)w.stl, (const int64_t*)w.meta,
                       (const int64_t*)w.pre[0], (const int64_t*)w.pre[kNodeScan], w.nbt, a.n_leaves / 8,
                       w.ntab, w.ncap);
  }
  if (w.ccap > 0) {
    int64_t rblocks = (w.ccap + 255) / 256;
    if (OC_TREE_TABLE_BLOCKS > 0 && rblocks > (int64_t)OC_TREE_TABLE_BLOCKS * L.num_cus)
      rblocks = (int64_t)OC_TREE_TABLE_BLOCKS * L.num_cus;
    hipLaunchKernelGGL(k_region_codes, dim3((unsigned)rblocks, w.ccap < 65536 ? kSets : 1),
                       dim3(256), 0, s,
                       a.trees, a.prefix, a.gd, a.gh, a.gw, a.n_leaves, (const int64_t*)w.bkey,
                       (const int32_t*)w.brow, (const int64_t*)w.meta,
                       (const int64_t*)w.pre[kSlotScan], w.cap, w.ccap, w.codes, w.smask);
  }
  return hipGetLastError();
}

bool conv_runs_fused(const ConvArgs& a, int impl) {
  if (impl != 2) return false;
  const MfmaVariant* v = find_variant(a.cin, a.cout);
  if (v == nullptr && conv_blocks(a.cin, a.cout).v == nullptr) return false;
  // The MFMA kernels gather input rows by a 32-bit row index (every
  // n_leaves < 2^31 the convolution accepts) with 16-byte loads.
  return (reinterpret_cast<uintptr_t>(a.in) & 15) == 0 && a.n_leaves < (int64_t)kNoRow;
}

hipError_t launch_conv_execute(const ConvArgs& a, void* ws, int impl, hipStream_t s) {
  const ConvWs w = carve(ws, a.n_trees, a.n_leaves, a.cin, a.cout, a.slot_cap);
  // Where the MFMA kernels cannot gather the input, the generic kernel (or,
  // for channel blocks, the GEMM path) runs.
  const MfmaVariant* v = find_variant(a.cin, a.cout);
  if (impl == 2 && !conv_runs_fused(a, impl)) impl = v ? 1 : 3;
  // Cell sums come from the fused kernels' epilogues only.
  if (a.sum_cells && impl != 2) return hipErrorInvalidValue;
  const uint32_t n_rows = (uint32_t)a.n_leaves;
  const int tm = generic_tile(a.cin);
  const size_t gsmem = generic_smem(a.cin, tm);
  const int64_t all_tiles = (a.n_leaves + tm - 1) / tm;
  if (impl != 2) {
    // The generic kernel and the window sums of the GEMM path locate every
    // leaf through the leaf index (the fused kernels need none).
    hipError_t e = launch_leaf_index(a.trees, a.prefix, a.n_trees, w.info, s);
    if (e != hipSuccess) return e;
  }
  if (impl == 3)
    return launch_conv_gemm(a, w.info, w.wt, w.sgemm, w.nbt, w.pre[0], (const int64_t*)(w.pre[0] + a.n_trees),
                            s);
  if (impl != 2) {
    const unsigned blocks = (unsigned)(all_tiles < 65536 ? all_tiles : 65536);
    hipLaunchKernelGGL(k_conv_generic, dim3(blocks), dim3(kThreads), gsmem, s, a.trees, a.prefix,
                       w.info, a.n_leaves, a.gd, a.gh, a.gw, a.in, a.cin, w.wt, a.bias, a.cout,
                       a.relu, a.out, tm, (const int32_t*)nullptr, (const int64_t*)nullptr);
    return hipGetLastError();
  }
  DevLimits L;
  hipError_t e = device_limits(&L);
  if (e != hipSuccess) return e;
  const int num_cus = L.num_cus;
  if (v != nullptr) {
    const FusedOut o{w.wm, w.wc, w.w8, a.bias, a.cout, a.relu | (a.sum_cells ? 2 : 0), a.out};
    return fused_pass(a, w, v, a.in, n_rows, o, 1, L, s);
  }
  // Channel blocks: per input block j (copied to a dense [n_leaves][32]
  // array unless it is the whole input), the boundary sums once, the K
  // output blocks' kernels into the partials, and their sum into the output.
  const Blocks bl = conv_blocks(a.cin, a.cout);
  if (bl.v == nullptr || bl.K > kMaxOutBlocks) return hipErrorInvalidValue;
  const int64_t n = a.n_leaves;
  for (int j = 0; j < bl.J; ++j) {
    const float* xin = a.in;
    if (bl.J > 1) {
      int64_t nb = (n * 8 + 255) / 256;
      if (nb > 8LL * num_cus * 8) nb = 8LL * num_cus * 8;
      hipLaunchKernelGGL(k_channel_block, dim3((unsigned)nb), dim3(256), 0, s, a.in, a.cin, j, n, w.xblk);
      xin = w.xblk;
    }
    // The K output blocks of input block j in one grid (rows k).
    const size_t b = (size_t)j * bl.K;
    const FusedOut o{w.wm + b * bl.v->wfloats, w.wc + b * bl.v->cell_wfloats, w.w8 + b * bl.v->wfloats,
                     nullptr, bl.cb, a.sum_cells ? 2 : 0, w.part};
    e = fused_pass(a, w, bl.v, xin, n_rows, o, bl.K, L, s);
    if (e != hipSuccess) return e;
    int64_t rb = (n * a.cout + 255) / 256;
    if (rb > 8LL * num_cus * 8) rb = 8LL * num_cus * 8;
    hipLaunchKernelGGL(k_block_accum, dim3((unsigned)rb), dim3(256), 0, s, (const float*)w.part, bl.K, bl.cb, n,
                       a.bias, j == 0 ? 1 : 0, j + 1 == bl.J ? 1 : 0, a.relu, a.out);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace oci

// The window-sum GEMM path for channel counts without a fused variant, and
// the gradients, in one translation unit with the forward kernels whose
// helpers and preparation they use.
#include "oc_conv_gemm.inc"
#include "oc_conv_bwd.inc"
