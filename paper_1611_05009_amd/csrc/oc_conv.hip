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
#include "oc_internal.h"

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
__constant__ int c_slot_off[27];
constexpr int kSlots = 6 * 64 + 12 * 8 + 8 + 1;  // 489
constexpr int kSelfSlot = kSlots - 1;

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
      cnt = enumerate_region(g, r, trees, prefix, gd, gh, gw, slots + c_slot_off[r]);
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
      const Entry* es = slots + (r == 13 ? kSelfSlot : c_slot_off[r]);
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
// Generic kernel: tile of `tm` consecutive rows per block.  Waves compute
// window sums into LDS, then all threads run the VALU contraction.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kThreads) k_conv_generic(
    const uint32_t* __restrict__ trees, const int64_t* __restrict__ prefix,
    const uint64_t* __restrict__ info, int64_t n_leaves, int gd, int gh, int gw,
    const float* __restrict__ in, int cin, const float* __restrict__ wt,
    const float* __restrict__ bias, int cout, int relu, float* __restrict__ out, int tm) {
  extern __shared__ float smem[];
  // layout: [4 waves][kSlots] entries, [4][27] counts, [tm][27*cin] sums, [tm] scale
  Entry* slots_all = reinterpret_cast<Entry*>(smem);
  int* counts_all = reinterpret_cast<int*>(slots_all + 4 * kSlots);
  float* sums = reinterpret_cast<float*>(counts_all + 4 * 32);
  float* scale = sums + (int64_t)tm * 27 * cin;
  const int wv = threadIdx.x >> 6;
  const int64_t row_base = (int64_t)blockIdx.x * tm;
  for (int m = wv; m < tm; m += 4) {
    const int64_t row = row_base + m;
    if (row < n_leaves) {
      const LeafGeo g = leaf_geo(info[row], row, gd, gh, gw);
      window_sums(g, trees, prefix, gd, gh, gw, in, cin, slots_all + wv * kSlots,
                  counts_all + wv * 32, sums + (int64_t)m * 27 * cin);
      if (lane_id() == 0) scale[m] = 1.f / (float)(g.s * g.s * g.s);
    }
    __builtin_amdgcn_wave_barrier();
  }
  __syncthreads();
  const int K = 27 * cin;
  for (int idx = threadIdx.x; idx < tm * cout; idx += kThreads) {
    const int m = idx / cout, co = idx % cout;
    const int64_t row = row_base + m;
    if (row >= n_leaves) continue;
    const float* sm = sums + (int64_t)m * K;
    float acc = 0.f;
    for (int k = 0; k < K; ++k) acc = fmaf(sm[k], wt[(int64_t)k * cout + co], acc);
    float v = acc * scale[m] + (bias ? bias[co] : 0.f);
    if (relu) v = fmaxf(v, 0.f);
    out[row * cout + co] = v;
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
  return sizeof(Entry) * 4 * kSlots + sizeof(int) * 4 * 32 + sizeof(float) * (size_t)tm * 27 * cin +
         sizeof(float) * tm;
}

bool g_slots_ready = false;

hipError_t init_slots() {
  if (g_slots_ready) return hipSuccess;
  int off[27];
  int acc = 0;
  for (int r = 0; r < 27; ++r) {
    off[r] = acc;
    if (r == 13) continue;
    const int dd = r / 9 - 1, dh = (r / 3) % 3 - 1, dw = r % 3 - 1;
    acc += (dd == 0 ? 8 : 1) * (dh == 0 ? 8 : 1) * (dw == 0 ? 8 : 1);
  }
  hipError_t e = hipMemcpyToSymbol(HIP_SYMBOL(c_slot_off), off, sizeof(off));
  if (e == hipSuccess) g_slots_ready = true;
  return e;
}

}  // namespace

namespace oci {

size_t conv_workspace(int64_t n_trees, int64_t n_leaves, int cin, int cout) {
  (void)n_trees;
  return align256(sizeof(uint64_t) * (size_t)n_leaves) + align256(sizeof(float) * 27 * (size_t)cin * cout) +
         256;
}

bool conv_mfma_supported(int cin, int cout) {
  (void)cin;
  (void)cout;
  return false;
}

// Workspace: [leaf_info: n_leaves x u64 | transposed weights: 27 cin cout f32]
hipError_t launch_conv_prepare(const ConvArgs& a, void* ws, hipStream_t s) {
  hipError_t e = init_slots();
  if (e != hipSuccess) return e;
  char* p = static_cast<char*>(ws);
  uint64_t* info = reinterpret_cast<uint64_t*>(p);
  p += align256(sizeof(uint64_t) * (size_t)a.n_leaves);
  float* wt = reinterpret_cast<float*>(p);
  e = launch_leaf_index(a.trees, a.prefix, a.n_trees, info, s);
  if (e != hipSuccess) return e;
  const int64_t nw = 27LL * a.cin * a.cout;
  hipLaunchKernelGGL(k_transpose_weights, dim3((unsigned)((nw + 255) / 256)), dim3(256), 0, s,
                     a.weight, a.cin, a.cout, wt);
  return hipGetLastError();
}

hipError_t launch_conv_execute(const ConvArgs& a, const void* ws, int impl, hipStream_t s) {
  (void)impl;
  hipError_t e = init_slots();
  if (e != hipSuccess) return e;
  const char* p = static_cast<const char*>(ws);
  const uint64_t* info = reinterpret_cast<const uint64_t*>(p);
  p += align256(sizeof(uint64_t) * (size_t)a.n_leaves);
  const float* wt = reinterpret_cast<const float*>(p);
  const int tm = generic_tile(a.cin);
  const size_t smem = generic_smem(a.cin, tm);
  const int64_t blocks = (a.n_leaves + tm - 1) / tm;
  hipLaunchKernelGGL(k_conv_generic, dim3((unsigned)blocks), dim3(kThreads), smem, s, a.trees,
                     a.prefix, info, a.n_leaves, a.gd, a.gh, a.gw, a.in, a.cin, wt, a.bias, a.cout,
                     a.relu, a.out, tm);
  return hipGetLastError();
}

}  // namespace oci
