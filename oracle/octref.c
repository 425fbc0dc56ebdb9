/*
 * octref.c -- CPU oracle for the grid-octree convolution hot path of
 * OctNet (Riegler, Ulusoy, Geiger, CVPR 2017).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain reference that the
 * GPU library is checked against.  Only the test-suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it.  It shares no code,
 * header, table or helper with the HIP library: every definition below is
 * re-derived from the paper's text.
 *
 * Floating point is double throughout (the paper fixes no precision).
 *
 * Conventions (readings of points the paper leaves open; each one is listed
 * in the design notes):
 *   - A shallow octree has depth 3 and covers 8x8x8 voxels (Sec. 3.1).
 *   - Bit j of a tree (0 <= j < 73) is stored in word j>>5 at position j&31
 *     of four uint32 words; bits 73..127 are zero.  Bit indices 73..584 name
 *     the implicit depth-3 voxels (children of depth-2 nodes, Eq. 2).
 *   - The child with octant o of a node covers the sub-cube whose offset along
 *     (d,h,w) is ((o>>2)&1, (o>>1)&1, o&1) times the child size.
 *   - Trees of the grid are concatenated in (n,d,h,w) order, w fastest; the
 *     leaves of one tree are stored in ascending bit-index (breadth-first)
 *     order (Sec. 3.1 and the supplement's "Data Index" section).
 *   - Voxels outside the D x H x W tree grid read as zero (zero padding).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define NBITS 73      /* stored split bits per shallow octree (Sec. 3.1) */
#define NNODES 585    /* 1 + 8 + 64 + 512 nodes of a depth-3 octree */

/* ------------------------------------------------------------------------- */
/* Bit strings and index arithmetic (Sec. 3.1, Eq. 1-3)                       */
/* ------------------------------------------------------------------------- */

/* Eq. 1: parent bit index. Defined for i >= 1. */
int ocref_parent(int i) { return (i - 1) / 8; }

/* Eq. 2: bit index of the first child. */
int ocref_child(int i) { return 8 * i + 1; }

/* Value of split bit i of a tree stored as four little-endian uint32 words.
 * Depth-3 voxels (i >= 73) are never split. */
int ocref_bit(const uint32_t *t, int i) {
  if (i < 0 || i >= NBITS) return 0;
  return (int)((t[i >> 5] >> (i & 31)) & 1u);
}

/* Depth of the node with bit index i in a tree with branching factor b. */
static int depth_of(int i, int b) {
  int d = 0, first = 0, cnt = 1;
  while (i >= first + cnt) { first += cnt; cnt *= b; d++; }
  return d;
}

/* Eq. 3, written for a general branching factor b (b = 8 for octrees; the
 * supplement's worked example uses the quadtree form with b = 4).
 * bits01[j] in {0,1} for j < nbits, and bits beyond nbits read as 0.
 * For i = 0 the formula is undefined (it would need pa(0)); the root, if it
 * is a leaf, is the only leaf, so data_idx(0) = 0. */
long ocref_data_idx_eq3(const uint8_t *bits01, int nbits, int b, int i) {
  if (i == 0) return 0;
  int pa = (i - 1) / b;
  long above = 0, before = 0;
  for (int j = 0; j < pa; ++j) above += (j < nbits) ? bits01[j] : 0;
  for (int j = 0; j < i; ++j) before += (j < nbits) ? bits01[j] : 0;
  long offset = (i - 1) % b; /* i >= 1 so this is the non-negative residue */
  return b * above + 1 - before + offset;
}

/* Data index by plain enumeration: the rank of leaf i among all leaves of the
 * tree taken in ascending bit index (breadth-first) order.  A node exists if
 * it is the root or its parent is split; it is a leaf if it exists and is
 * either at maximum depth or not split.  Returns -1 if i is not a leaf. */
long ocref_data_idx_bfs(const uint8_t *bits01, int nbits, int b, int maxdepth, int i) {
  long total = 0; /* number of nodes in a full tree of depth maxdepth */
  long cnt = 1;
  for (int d = 0; d <= maxdepth; ++d) { total += cnt; cnt *= b; }
  if (i < 0 || i >= total) return -1;
  uint8_t *exists = (uint8_t *)calloc((size_t)total, 1);
  exists[0] = 1;
  long rank = 0, result = -1;
  for (long j = 0; j < total; ++j) {
    if (j > 0) {
      long p = (j - 1) / b;
      int pbit = (p < nbits) ? bits01[p] : 0;
      exists[j] = exists[p] && pbit;
    }
    if (!exists[j]) continue;
    int bj = (j < nbits) ? bits01[j] : 0;
    int leaf = (depth_of((int)j, b) == maxdepth) || !bj;
    if (!leaf) continue;
    if (j == i) { result = rank; break; }
    rank++;
  }
  free(exists);
  return result;
}

/* Geometry of node i of an octree: depth, local origin (in voxels of the
 * 8^3 tree) and edge length.  Walks the octant path from i up to the root. */
static void node_geom(int i, int *depth, int *od, int *oh, int *ow, int *size) {
  int path[4], k = 0;
  while (i > 0) { path[k++] = (i - 1) % 8; i = (i - 1) / 8; }
  int s = 8, d = 0, h = 0, w = 0;
  for (int j = k - 1; j >= 0; --j) {
    s /= 2;
    int o = path[j];
    d += ((o >> 2) & 1) * s;
    h += ((o >> 1) & 1) * s;
    w += (o & 1) * s;
  }
  *depth = k; *od = d; *oh = h; *ow = w; *size = 8 >> k;
}

/* Does node i of tree t exist (root, or parent split)? */
static int node_exists(const uint32_t *t, int i) {
  while (i > 0) {
    int p = (i - 1) / 8;
    if (!ocref_bit(t, p)) return 0;
    i = p;
  }
  return 1;
}

static int node_is_leaf(const uint32_t *t, int i) {
  return node_exists(t, i) && (i >= NBITS || !ocref_bit(t, i));
}

/* Leaves of one tree in ascending bit index order; returns their number. */
static int tree_leaves(const uint32_t *t, int *out) {
  int n = 0;
  for (int i = 0; i < NNODES; ++i)
    if (node_is_leaf(t, i)) out[n++] = i;
  return n;
}

int ocref_tree_n_leaves(const uint32_t *t) {
  int tmp[NNODES];
  return tree_leaves(t, tmp);
}

/* Canonical form: no set bit below an unsplit node, no bit beyond 72. */
int ocref_tree_valid(const uint32_t *t) {
  if ((t[2] >> 9) != 0 || t[3] != 0) return 0;
  for (int i = 1; i < NBITS; ++i)
    if (ocref_bit(t, i) && !ocref_bit(t, (i - 1) / 8)) return 0;
  return 1;
}

static void set_bit(uint32_t *t, int i) { t[i >> 5] |= (1u << (i & 31)); }

/* ------------------------------------------------------------------------- */
/* Grid bookkeeping                                                           */
/* ------------------------------------------------------------------------- */

/* prefix[t] = number of leaves in trees 0..t-1; prefix[n_trees] = total. */
void ocref_prefix(const uint32_t *trees, long n_trees, int64_t *prefix) {
  prefix[0] = 0;
  for (long t = 0; t < n_trees; ++t)
    prefix[t + 1] = prefix[t] + ocref_tree_n_leaves(trees + 4 * t);
}

/* leaf_info[row] = tree << 10 | bit index, rows in concatenation order. */
void ocref_leaf_info(const uint32_t *trees, long n_trees, const int64_t *prefix,
                     uint64_t *leaf_info) {
#pragma omp parallel for schedule(dynamic, 64)
  for (long t = 0; t < n_trees; ++t) {
    int lv[NNODES];
    int n = tree_leaves(trees + 4 * t, lv);
    for (int k = 0; k < n; ++k)
      leaf_info[prefix[t] + k] = ((uint64_t)t << 10) | (uint64_t)lv[k];
  }
}

/* rowmap[n][8gd][8gh][8gw] = global row of the leaf that contains the voxel,
 * i.e. oc2ten (Eq. 4) applied to the row number instead of the feature. */
static void build_rowmap_sample(const uint32_t *trees, const int64_t *prefix,
                                int sample, int gd, int gh, int gw, int64_t *rowmap) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  long tree0 = (long)sample * gd * gh * gw;
#pragma omp parallel for collapse(3) schedule(static)
  for (int td = 0; td < gd; ++td)
    for (int th = 0; th < gh; ++th)
      for (int tw = 0; tw < gw; ++tw) {
        long t = tree0 + ((long)td * gh + th) * gw + tw;
        const uint32_t *bits = trees + 4 * t;
        int lv[NNODES];
        int n = tree_leaves(bits, lv);
        for (int k = 0; k < n; ++k) {
          int dep, od, oh, ow, s;
          node_geom(lv[k], &dep, &od, &oh, &ow, &s);
          for (int a = 0; a < s; ++a)
            for (int b = 0; b < s; ++b)
              for (int c = 0; c < s; ++c) {
                long vd = 8L * td + od + a, vh = 8L * th + oh + b, vw = 8L * tw + ow + c;
                rowmap[(vd * H + vh) * W + vw] = prefix[t] + k;
              }
        }
      }
  (void)D;
}

void ocref_rowmap(const uint32_t *trees, const int64_t *prefix, int n, int gd, int gh,
                  int gw, int64_t *rowmap) {
  long vox = 512L * gd * gh * gw;
  for (int s = 0; s < n; ++s)
    build_rowmap_sample(trees, prefix, s, gd, gh, gw, rowmap + s * vox);
}

/* ------------------------------------------------------------------------- */
/* Octree creation from a voxel occupancy grid (Sec. 1 and 3.1)               */
/* ------------------------------------------------------------------------- */

/* rule 0: split a node iff the occupancy inside it is mixed (some voxels
 *         occupied, some empty).
 * rule 1: split a node iff any voxel inside it is occupied.
 * Nodes are only considered when their parent is split. */
void ocref_build(const uint8_t *occ, int n, int gd, int gh, int gw, int rule,
                 uint32_t *trees) {
  long H = 8L * gh, W = 8L * gw, D = 8L * gd;
  long n_trees = (long)n * gd * gh * gw;
#pragma omp parallel for schedule(static)
  for (long t = 0; t < n_trees; ++t) {
    long rem = t;
    int tw = rem % gw; rem /= gw;
    int th = rem % gh; rem /= gh;
    int td = rem % gd; rem /= gd;
    int sample = (int)rem;
    const uint8_t *o = occ + (long)sample * D * H * W;
    uint32_t *bits = trees + 4 * t;
    bits[0] = bits[1] = bits[2] = bits[3] = 0;
    for (int i = 0; i < NBITS; ++i) {
      if (i > 0 && !ocref_bit(bits, (i - 1) / 8)) continue;
      int dep, od, oh, ow, s;
      node_geom(i, &dep, &od, &oh, &ow, &s);
      int any = 0, all = 1;
      for (int a = 0; a < s; ++a)
        for (int b = 0; b < s; ++b)
          for (int c = 0; c < s; ++c) {
            long vd = 8L * td + od + a, vh = 8L * th + oh + b, vw = 8L * tw + ow + c;
            int v = o[(vd * H + vh) * W + vw] != 0;
            any |= v;
            all &= v;
          }
      int split = rule == 0 ? (any && !all) : any;
      if (split) set_bit(bits, i);
    }
  }
}

/* ------------------------------------------------------------------------- */
/* oc2ten and ten2oc (Eq. 4 and Eq. 5)                                        */
/* ------------------------------------------------------------------------- */

/* dense[n][8gd][8gh][8gw][c] = data[row of containing leaf][c]  (Eq. 4). */
void ocref_oc2ten(const int64_t *rowmap, long n_vox, const double *data, int c,
                  double *dense) {
#pragma omp parallel for schedule(static)
  for (long v = 0; v < n_vox; ++v)
    for (int k = 0; k < c; ++k) dense[v * c + k] = data[rowmap[v] * c + k];
}

/* data[leaf][c] = pool over the leaf's cell of dense (Eq. 5).
 * pool 0 = average, 1 = max.  Sums are accumulated in double. */
void ocref_ten2oc(const uint32_t *trees, const int64_t *prefix, int n, int gd, int gh,
                  int gw, const double *dense, int c, int pool, double *data) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  long n_trees = (long)n * gd * gh * gw;
#pragma omp parallel for schedule(dynamic, 16)
  for (long t = 0; t < n_trees; ++t) {
    long rem = t;
    int tw = rem % gw; rem /= gw;
    int th = rem % gh; rem /= gh;
    int td = rem % gd; rem /= gd;
    long sample = rem;
    int lv[NNODES];
    int nl = tree_leaves(trees + 4 * t, lv);
    for (int k = 0; k < nl; ++k) {
      int dep, od, oh, ow, s;
      node_geom(lv[k], &dep, &od, &oh, &ow, &s);
      for (int ch = 0; ch < c; ++ch) {
        double acc = pool == 0 ? 0.0 : -INFINITY;
        for (int a = 0; a < s; ++a)
          for (int b = 0; b < s; ++b)
            for (int e = 0; e < s; ++e) {
              long vd = 8L * td + od + a, vh = 8L * th + oh + b, vw = 8L * tw + ow + e;
              double x = dense[(((sample * D + vd) * H + vh) * W + vw) * c + ch];
              if (pool == 0) acc += x;
              else if (x > acc) acc = x;
            }
        if (pool == 0) acc /= (double)s * s * s;
        data[(prefix[t] + k) * c + ch] = acc;
      }
    }
  }
}

/* ------------------------------------------------------------------------- */
/* Convolution on the grid-octree (Eq. 7 and Eq. 8)                           */
/* ------------------------------------------------------------------------- */

/* For each requested leaf, evaluate the dense 3x3x3 convolution of Eq. 7 at
 * every voxel of the leaf's cell, with the input read through oc2ten (Eq. 4)
 * and zero outside the grid, then average over the cell (Eq. 5 / Eq. 8 with
 * average pooling), add the bias and optionally clamp at zero.
 *
 *   w[co][ci][l][m][n]; the input voxel of tap (l,m,n) for output voxel
 *   (i,j,k) is (i-l+1, j-m+1, k-n+1)  -- Eq. 7 with L = M = N = 3.
 *
 * rowmap holds every sample (rm_sample < 0) or only sample rm_sample, in
 * which case every requested leaf must lie in that sample.
 * rows[r] lists the leaves to evaluate (global rows); leaf_info gives their
 * tree and bit index.  out[r][co] receives the result. */
void ocref_conv3(const uint32_t *trees, const uint64_t *leaf_info, const int64_t *rowmap,
                 int rm_sample, int n, int gd, int gh, int gw, const double *data, int cin,
                 const double *w, const double *bias, int cout, int relu,
                 const int64_t *rows, long n_rows, double *out) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  long trees_per_sample = (long)gd * gh * gw;
  (void)trees; (void)n;
#pragma omp parallel for schedule(dynamic, 4)
  for (long r = 0; r < n_rows; ++r) {
    uint64_t info = leaf_info[rows[r]];
    long t = (long)(info >> 10);
    int bit = (int)(info & 1023);
    long rem = t;
    int tw = rem % gw; rem /= gw;
    int th = rem % gh; rem /= gh;
    int td = rem % gd; rem /= gd;
    long sample = rem;
    if (rm_sample >= 0 && sample != rm_sample) {
      for (int co = 0; co < cout; ++co) out[r * cout + co] = NAN;
      continue;
    }
    const int64_t *rm = rm_sample >= 0 ? rowmap : rowmap + sample * D * H * W;
    (void)trees_per_sample;
    int dep, od, oh, ow, s;
    node_geom(bit, &dep, &od, &oh, &ow, &s);
    double *acc = (double *)calloc((size_t)cout, sizeof(double));
    for (int a = 0; a < s; ++a)
      for (int b = 0; b < s; ++b)
        for (int e = 0; e < s; ++e) {
          long i = 8L * td + od + a, j = 8L * th + oh + b, k = 8L * tw + ow + e;
          for (int l = 0; l < 3; ++l)
            for (int m = 0; m < 3; ++m)
              for (int q = 0; q < 3; ++q) {
                long ii = i - l + 1, jj = j - m + 1, kk = k - q + 1;
                if (ii < 0 || ii >= D || jj < 0 || jj >= H || kk < 0 || kk >= W) continue;
                const double *x = data + rm[(ii * H + jj) * W + kk] * cin;
                for (int co = 0; co < cout; ++co) {
                  const double *wc = w + (long)co * cin * 27 + (l * 9 + m * 3 + q);
                  double sum = 0.0;
                  for (int ci = 0; ci < cin; ++ci) sum += wc[ci * 27] * x[ci];
                  acc[co] += sum;
                }
              }
        }
    double vol = (double)s * s * s;
    for (int co = 0; co < cout; ++co) {
      double v = acc[co] / vol + (bias ? bias[co] : 0.0);
      if (relu && v < 0.0) v = 0.0;
      out[r * cout + co] = v;
    }
    free(acc);
  }
}

/* Dense 3x3x3 convolution of Eq. 7 over a whole NDHWC tensor with zero
 * padding 1 (used on tiny grids, where the oracle chains oc2ten -> this ->
 * ten2oc literally as Eq. 6). */
void ocref_dense_conv3(const double *x, int n, long D, long H, long W, int cin,
                       const double *w, int cout, double *y) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int s = 0; s < n; ++s)
    for (long i = 0; i < D; ++i)
      for (long j = 0; j < H; ++j)
        for (long k = 0; k < W; ++k) {
          double *yo = y + ((((long)s * D + i) * H + j) * W + k) * cout;
          for (int co = 0; co < cout; ++co) yo[co] = 0.0;
          for (int l = 0; l < 3; ++l)
            for (int m = 0; m < 3; ++m)
              for (int q = 0; q < 3; ++q) {
                long ii = i - l + 1, jj = j - m + 1, kk = k - q + 1;
                if (ii < 0 || ii >= D || jj < 0 || jj >= H || kk < 0 || kk >= W) continue;
                const double *xi = x + ((((long)s * D + ii) * H + jj) * W + kk) * cin;
                for (int co = 0; co < cout; ++co) {
                  double sum = 0.0;
                  for (int ci = 0; ci < cin; ++ci)
                    sum += w[((long)co * cin + ci) * 27 + l * 9 + m * 3 + q] * xi[ci];
                  yo[co] += sum;
                }
              }
        }
}

/* ------------------------------------------------------------------------- */
/* 2x2x2 pooling on the grid-octree (Eq. 9 and Eq. 10)                        */
/* ------------------------------------------------------------------------- */

/* Output structure: input trees (2d+a, 2h+b, 2w+c) form octant o = 4a+2b+c of
 * output tree (d,h,w).  Every input node moves one level deeper: input node
 * at depth k with in-tree index p becomes the output node reached from
 * output child o by the same octant path.  The output root is always split;
 * input depth-2 split bits have no place in the output (their children,
 * the depth-3 voxels, are max-pooled by Eq. 10). */
void ocref_pool2_structure(const uint32_t *in_trees, int n, int gd, int gh, int gw,
                           uint32_t *out_trees) {
  int od = gd / 2, oh = gh / 2, ow = gw / 2;
  long n_out = (long)n * od * oh * ow;
#pragma omp parallel for schedule(static)
  for (long t = 0; t < n_out; ++t) {
    long rem = t;
    int w = rem % ow; rem /= ow;
    int h = rem % oh; rem /= oh;
    int d = rem % od; rem /= od;
    long sample = rem;
    uint32_t *bits = out_trees + 4 * t;
    bits[0] = bits[1] = bits[2] = bits[3] = 0;
    set_bit(bits, 0);
    for (int o = 0; o < 8; ++o) {
      int a = (o >> 2) & 1, b = (o >> 1) & 1, c = o & 1;
      long ti = ((sample * gd + 2 * d + a) * gh + 2 * h + b) * gw + 2 * w + c;
      const uint32_t *ib = in_trees + 4 * ti;
      /* input node p at depth 0 or 1 -> output node at depth 1 or 2 */
      if (ocref_bit(ib, 0)) set_bit(bits, 1 + o);
      for (int q = 0; q < 8; ++q)
        if (ocref_bit(ib, 1 + q)) set_bit(bits, 9 + 8 * o + q);
    }
  }
}

/* Value of the grid-octree at a global voxel (Eq. 4) plus the depth of the
 * containing leaf. */
static double oc_value(const int64_t *rm, long H, long W, const uint64_t *leaf_info,
                       const double *data, int c, int ch, long i, long j, long k,
                       int *depth) {
  long row = rm[(i * H + j) * W + k];
  if (depth) {
    int bit = (int)(leaf_info[row] & 1023), dep, a, b, e, s;
    node_geom(bit, &dep, &a, &b, &e, &s);
    *depth = dep;
  }
  return data[row * c + ch];
}

/* Output data by Eq. 10, evaluated at the first voxel of each output leaf:
 *   O_out[i,j,k] = O_in[2i,2j,2k]                      if depth(2i,2j,2k) < 3
 *                = max over l,m,n in {0,1} of O_in[2i+l,2j+m,2k+n]  otherwise. */
void ocref_pool2_max(const uint64_t *in_leaf_info, const int64_t *in_rowmap, int n,
                     int gd, int gh, int gw, const double *in_data, int c,
                     const uint64_t *out_leaf_info, long out_rows, double *out_data) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  int ogd = gd / 2, ogh = gh / 2, ogw = gw / 2;
  (void)n;
#pragma omp parallel for schedule(static)
  for (long r = 0; r < out_rows; ++r) {
    long t = (long)(out_leaf_info[r] >> 10);
    int bit = (int)(out_leaf_info[r] & 1023);
    long rem = t;
    int tw = rem % ogw; rem /= ogw;
    int th = rem % ogh; rem /= ogh;
    int td = rem % ogd; rem /= ogd;
    long sample = rem;
    const int64_t *rm = in_rowmap + sample * D * H * W;
    int dep, od, oh, ow, s;
    node_geom(bit, &dep, &od, &oh, &ow, &s);
    long i = 8L * td + od, j = 8L * th + oh, k = 8L * tw + ow;
    for (int ch = 0; ch < c; ++ch) {
      int vd;
      double v = oc_value(rm, H, W, in_leaf_info, in_data, c, ch, 2 * i, 2 * j, 2 * k, &vd);
      if (vd >= 3) {
        for (int l = 0; l < 2; ++l)
          for (int m = 0; m < 2; ++m)
            for (int q = 0; q < 2; ++q) {
              double x = oc_value(rm, H, W, in_leaf_info, in_data, c, ch, 2 * i + l,
                                  2 * j + m, 2 * k + q, NULL);
              if (x > v) v = x;
            }
      }
      out_data[r * c + ch] = v;
    }
  }
}

/* ------------------------------------------------------------------------- */
/* 2x2x2 unpooling on the grid-octree (Eq. 11 and Eq. 12, and the guided     */
/* variant of the remark that follows Eq. 12)                                 */
/* ------------------------------------------------------------------------- */

/* Plain unpooling structure: input tree (d,h,w) spawns output trees
 * (2d+a, 2h+b, 2w+c), o = 4a+2b+c.  If the input root is not split the whole
 * tree is one cell and every spawned tree is an unsplit root.  Otherwise
 * input node 1+o becomes the root of output tree o and every node below it
 * moves one level up (its size in output voxels stays twice its input size,
 * which is the same fraction of the new tree). */
void ocref_unpool2_structure(const uint32_t *in_trees, int n, int gd, int gh, int gw,
                             uint32_t *out_trees) {
  int Gd = 2 * gd, Gh = 2 * gh, Gw = 2 * gw;
  long n_out = (long)n * Gd * Gh * Gw;
#pragma omp parallel for schedule(static)
  for (long t = 0; t < n_out; ++t) {
    long rem = t;
    int w = rem % Gw; rem /= Gw;
    int h = rem % Gh; rem /= Gh;
    int d = rem % Gd; rem /= Gd;
    long sample = rem;
    int o = ((d & 1) << 2) | ((h & 1) << 1) | (w & 1);
    long ti = ((sample * gd + d / 2) * gh + h / 2) * gw + w / 2;
    const uint32_t *ib = in_trees + 4 * ti;
    uint32_t *bits = out_trees + 4 * t;
    bits[0] = bits[1] = bits[2] = bits[3] = 0;
    if (ocref_bit(ib, 0) && ocref_bit(ib, 1 + o)) {
      set_bit(bits, 0);
      for (int q = 0; q < 8; ++q)
        if (ocref_bit(ib, 9 + 8 * o + q)) set_bit(bits, 1 + q);
    }
  }
}

/* Unpooled data by Eq. 12 evaluated at the first voxel of each output leaf:
 *   O_out[i,j,k] = O_in[floor(i/2), floor(j/2), floor(k/2)].
 * The same rule gives the guided variant, whose output structure is the
 * guide: every guide leaf takes the coarse value that covers it. */
void ocref_unpool2(const int64_t *in_rowmap, int gd, int gh, int gw, const double *in_data,
                   int c, const uint64_t *out_leaf_info, long out_rows, double *out_data) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  int Gd = 2 * gd, Gh = 2 * gh, Gw = 2 * gw;
#pragma omp parallel for schedule(static)
  for (long r = 0; r < out_rows; ++r) {
    long t = (long)(out_leaf_info[r] >> 10);
    int bit = (int)(out_leaf_info[r] & 1023);
    long rem = t;
    int tw = rem % Gw; rem /= Gw;
    int th = rem % Gh; rem /= Gh;
    int td = rem % Gd; rem /= Gd;
    long sample = rem;
    const int64_t *rm = in_rowmap + sample * D * H * W;
    int dep, od, oh, ow, s;
    node_geom(bit, &dep, &od, &oh, &ow, &s);
    long i = 8L * td + od, j = 8L * th + oh, k = 8L * tw + ow;
    long row = rm[((i / 2) * H + j / 2) * W + k / 2];
    for (int ch = 0; ch < c; ++ch) out_data[r * c + ch] = in_data[row * c + ch];
  }
}

/* ------------------------------------------------------------------------- */
/* Gradients (backward passes) of the convolution, pooling and unpooling.     */
/* Each is the adjoint of the forward map as the forward is defined above:    */
/* the convolution of Eq. 8 is linear in the input and in the weights, pool   */
/* (Eq. 10) selects one input value per output value, unpool (Eq. 12) copies. */
/* ------------------------------------------------------------------------- */

static double leaf_volume(const uint64_t *leaf_info, long row) {
  int dep, a, b, e, s;
  node_geom((int)(leaf_info[row] & 1023), &dep, &a, &b, &e, &s);
  return (double)s * s * s;
}

/* Input gradient of Eq. 8 (bias and ReLU excluded).  Output voxel v of leaf l
 * receives dy[l] / |l| (the average of Eq. 8 spreads it over the cell), and
 * reads input voxel v - (tap - 1) with tap weight W[co][ci][tap] (Eq. 7).
 * So input voxel u collects sum over taps of W^T dy[leaf(u + tap - 1)] /
 * |leaf(u + tap - 1)|, and input leaf l' sums that over its voxels.
 * rowmap holds every sample; dx [n_leaves][cin] is overwritten. */
void ocref_conv3_bwd_data(const uint64_t *leaf_info, const int64_t *rowmap, int n, int gd,
                          int gh, int gw, const double *dy, int cout, const double *w, int cin,
                          long n_leaves, double *dx) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  (void)n;
#pragma omp parallel for schedule(dynamic, 4)
  for (long r = 0; r < n_leaves; ++r) {
    uint64_t info = leaf_info[r];
    long t = (long)(info >> 10);
    int bit = (int)(info & 1023);
    long rem = t;
    int tw = rem % gw; rem /= gw;
    int th = rem % gh; rem /= gh;
    int td = rem % gd; rem /= gd;
    long sample = rem;
    const int64_t *rm = rowmap + sample * D * H * W;
    int dep, od, oh, ow, s;
    node_geom(bit, &dep, &od, &oh, &ow, &s);
    double *acc = dx + r * cin;
    for (int ci = 0; ci < cin; ++ci) acc[ci] = 0.0;
    for (int a = 0; a < s; ++a)
      for (int b = 0; b < s; ++b)
        for (int e = 0; e < s; ++e) {
          long i = 8L * td + od + a, j = 8L * th + oh + b, k = 8L * tw + ow + e;
          for (int l = 0; l < 3; ++l)
            for (int m = 0; m < 3; ++m)
              for (int q = 0; q < 3; ++q) {
                long vi = i + l - 1, vj = j + m - 1, vk = k + q - 1;  /* output voxel */
                if (vi < 0 || vi >= D || vj < 0 || vj >= H || vk < 0 || vk >= W) continue;
                long ol = rm[(vi * H + vj) * W + vk];
                double inv = 1.0 / leaf_volume(leaf_info, ol);
                const double *g = dy + ol * cout;
                for (int ci = 0; ci < cin; ++ci) {
                  double sum = 0.0;
                  for (int co = 0; co < cout; ++co)
                    sum += w[((long)co * cin + ci) * 27 + l * 9 + m * 3 + q] * g[co];
                  acc[ci] += sum * inv;
                }
              }
        }
  }
}

/* Weight and bias gradients of Eq. 8: dw[co][ci][tap] = sum over leaves l of
 * dy[l][co] / |l| times the sum over l's voxels v of x at v - (tap - 1)
 * (zero outside the grid); db[co] = sum over leaves of dy[l][co].  Summed in
 * row order, one output channel per thread. */
void ocref_conv3_bwd_weight(const uint64_t *leaf_info, const int64_t *rowmap, int n, int gd,
                            int gh, int gw, const double *x, int cin, const double *dy, int cout,
                            long n_leaves, double *dw, double *db) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  (void)n;
#pragma omp parallel for schedule(dynamic, 1)
  for (int co = 0; co < cout; ++co) {
    double *dwc = dw + (long)co * cin * 27;
    for (long z = 0; z < (long)cin * 27; ++z) dwc[z] = 0.0;
    double bsum = 0.0;
    for (long r = 0; r < n_leaves; ++r) {
      uint64_t info = leaf_info[r];
      long t = (long)(info >> 10);
      int bit = (int)(info & 1023);
      long rem = t;
      int tw = rem % gw; rem /= gw;
      int th = rem % gh; rem /= gh;
      int td = rem % gd; rem /= gd;
      long sample = rem;
      const int64_t *rm = rowmap + sample * D * H * W;
      int dep, od, oh, ow, s;
      node_geom(bit, &dep, &od, &oh, &ow, &s);
      double g = dy[r * cout + co];
      bsum += g;
      g /= (double)s * s * s;
      for (int a = 0; a < s; ++a)
        for (int b = 0; b < s; ++b)
          for (int e = 0; e < s; ++e) {
            long i = 8L * td + od + a, j = 8L * th + oh + b, k = 8L * tw + ow + e;
            for (int l = 0; l < 3; ++l)
              for (int m = 0; m < 3; ++m)
                for (int q = 0; q < 3; ++q) {
                  long ii = i - l + 1, jj = j - m + 1, kk = k - q + 1;
                  if (ii < 0 || ii >= D || jj < 0 || jj >= H || kk < 0 || kk >= W) continue;
                  const double *xi = x + rm[(ii * H + jj) * W + kk] * cin;
                  for (int ci = 0; ci < cin; ++ci) dwc[(long)ci * 27 + l * 9 + m * 3 + q] += g * xi[ci];
                }
          }
    }
    db[co] = bsum;
  }
}

/* Gradient of Eq. 10: an output value that copies an input cell passes its
 * gradient to that cell; one that is the maximum of 8 depth-3 voxels passes
 * it to the first of them (order l, m, n) that attains the maximum, per
 * channel.  dx [in_rows][c] is overwritten. */
void ocref_pool2_max_bwd(const uint64_t *in_leaf_info, const int64_t *in_rowmap, int n,
                         int gd, int gh, int gw, const double *in_data, int c,
                         const uint64_t *out_leaf_info, long out_rows, const double *dy,
                         long in_rows, double *dx) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  int ogd = gd / 2, ogh = gh / 2, ogw = gw / 2;
  (void)n;
  for (long z = 0; z < in_rows * c; ++z) dx[z] = 0.0;
  for (long r = 0; r < out_rows; ++r) {
    long t = (long)(out_leaf_info[r] >> 10);
    int bit = (int)(out_leaf_info[r] & 1023);
    long rem = t;
    int tw = rem % ogw; rem /= ogw;
    int th = rem % ogh; rem /= ogh;
    int td = rem % ogd; rem /= ogd;
    long sample = rem;
    const int64_t *rm = in_rowmap + sample * D * H * W;
    int dep, od, oh, ow, s;
    node_geom(bit, &dep, &od, &oh, &ow, &s);
    long i = 2 * (8L * td + od), j = 2 * (8L * th + oh), k = 2 * (8L * tw + ow);
    for (int ch = 0; ch < c; ++ch) {
      int vd;
      double v = oc_value(rm, H, W, in_leaf_info, in_data, c, ch, i, j, k, &vd);
      long best = rm[(i * H + j) * W + k];
      if (vd >= 3) {
        for (int l = 0; l < 2; ++l)
          for (int m = 0; m < 2; ++m)
            for (int q = 0; q < 2; ++q) {
              double xv = oc_value(rm, H, W, in_leaf_info, in_data, c, ch, i + l, j + m, k + q, NULL);
              if (xv > v) {
                v = xv;
                best = rm[((i + l) * H + j + m) * W + k + q];
              }
            }
      }
      dx[best * c + ch] += dy[r * c + ch];
    }
  }
}

/* Gradient of Eq. 12 (plain or guided): every output leaf copies the input
 * leaf holding floor(v / 2) of its first voxel v, so that input leaf sums
 * the gradients of all output leaves that copy it, in output row order.
 * dx [in_rows][c] is overwritten. */
void ocref_unpool2_bwd(const int64_t *in_rowmap, int gd, int gh, int gw, int c,
                       const uint64_t *out_leaf_info, long out_rows, const double *dy,
                       long in_rows, double *dx) {
  long D = 8L * gd, H = 8L * gh, W = 8L * gw;
  int Gd = 2 * gd, Gh = 2 * gh, Gw = 2 * gw;
  for (long z = 0; z < in_rows * c; ++z) dx[z] = 0.0;
  for (long r = 0; r < out_rows; ++r) {
    long t = (long)(out_leaf_info[r] >> 10);
    int bit = (int)(out_leaf_info[r] & 1023);
    long rem = t;
    int tw = rem % Gw; rem /= Gw;
    int th = rem % Gh; rem /= Gh;
    int td = rem % Gd; rem /= Gd;
    long sample = rem;
    const int64_t *rm = in_rowmap + sample * D * H * W;
    int dep, od, oh, ow, s;
    node_geom(bit, &dep, &od, &oh, &ow, &s);
    long i = 8L * td + od, j = 8L * th + oh, k = 8L * tw + ow;
    long row = rm[((i / 2) * H + j / 2) * W + k / 2];
    for (int ch = 0; ch < c; ++ch) dx[row * c + ch] += dy[r * c + ch];
  }
}

/* Element-wise rectifier (pointwise ops act on leaf data unchanged, Sec. 3.2). */
void ocref_relu(double *x, long count) {
  for (long i = 0; i < count; ++i)
    if (x[i] < 0.0) x[i] = 0.0;
}

int ocref_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void ocref_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
