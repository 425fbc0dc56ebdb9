/*
 * octnet_hip.h -- C ABI of the MI355X (gfx950) grid-octree library.
 *
 * Implements the hot path of OctNet (Riegler, Ulusoy, Geiger, "OctNet:
 * Learning Deep 3D Representations at High Resolutions", CVPR 2017):
 * the hybrid grid-octree of Sec. 3.1 and the convolution, pooling and
 * unpooling of Sec. 3.2, all run by hand-written HIP kernels.
 *
 * Data layout (shared by every call):
 *   - A batch of n grids, each of gd x gh x gw shallow octrees of depth 3,
 *     covers a voxel grid of 8gd x 8gh x 8gw (Sec. 3.1).
 *   - trees: uint32 [n_trees][4], n_trees = n*gd*gh*gw, trees ordered
 *     (n, d, h, w) with w fastest.  Split bit j (0 <= j < 73, Sec. 3.1) is
 *     (trees[4t + (j>>5)] >> (j&31)) & 1; bits 73..127 are 0.  Bit 0 is the
 *     root, bits 1..8 depth 1, bits 9..72 depth 2; bit indices 73..584 name
 *     the implicit depth-3 voxels.  parent(i) = (i-1)/8 and child(i) = 8i+1
 *     (Eq. 1-2).  The child with octant o covers the sub-cube offset by
 *     ((o>>2)&1, (o>>1)&1, o&1) times the child size along (d, h, w).
 *   - A tree is canonical when no bit is set below an unsplit node.  Every
 *     call below assumes canonical trees.  oc_build and the pooling and
 *     unpooling structure calls only produce canonical trees; oc_prefix,
 *     where trees made elsewhere enter, rejects non-canonical ones with
 *     OC_ESTRUCT; oc_validate (device) and oc_validate_host (host, header
 *     only) check explicitly.
 *   - prefix: int64 [n_trees + 1], prefix[t] = leaves in trees 0..t-1.  The
 *     leaves of tree t occupy rows prefix[t] .. prefix[t+1]-1 in ascending
 *     bit-index order, i.e. row = prefix[t] + data_idx(i) with data_idx from
 *     Eq. 3.
 *   - Leaf features: float [n_leaves][c], row-major.
 *   - Dense tensors: float [n][8gd][8gh][8gw][c] (NDHWC).
 *
 * Conventions: every pointer is a device pointer unless marked [host].
 * `stream` is a hipStream_t (NULL = the default stream).  Calls are
 * asynchronous on that stream except where marked "synchronizes".  The caller
 * owns every buffer; no call allocates or frees device memory.  Outputs must
 * not alias inputs (except oc_relu and oc_relu_backward).  Argument errors are detected on the host
 * before any launch and leave every buffer untouched.
 */
#ifndef OCTNET_HIP_H
#define OCTNET_HIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define OC_OK 0
#define OC_EINVAL (-1)      /* null pointer, non-positive size, odd dims for pooling, ... */
#define OC_ESTRUCT (-2)     /* non-canonical tree, or a guide that does not pool to the input */
#define OC_EWORKSPACE (-3)  /* workspace smaller than the matching *_workspace query */
#define OC_EHIP (-4)        /* HIP runtime or launch failure; see oc_last_error() */
#define OC_EOVERFLOW (-5)   /* a count exceeds what the layout supports */

/* Split rules of oc_build. */
#define OC_SPLIT_MIXED 0 /* split a node iff its occupancy is mixed */
#define OC_SPLIT_ANY 1   /* split a node iff any voxel in it is occupied */

/* Pooling functions of oc_ten2oc (Eq. 5). */
#define OC_POOL_AVG 0
#define OC_POOL_MAX 1

/* Convolution implementations (oc_conv3x3x3_ex). */
#define OC_CONV_AUTO 0    /* OC_CONV_MFMA where a fused variant exists, or in channel blocks on >= 65536 leaves (>= 16384 for cin >= 128); else OC_CONV_GEMM */
#define OC_CONV_GENERIC 1 /* any channel counts: window sums + VALU contraction */
#define OC_CONV_MFMA 2    /* fused fp32 MFMA kernels; OC_EINVAL if unsupported */
#define OC_CONV_GEMM 3    /* any channel counts: window sums of row chunks, then an fp32 MFMA GEMM */
#define OC_CONV_TRUNCATED 4 /* the supplement's efficient convolution (constant part + truncated
                              kernels at boundary voxels), VALU; oc_conv3x3x3_ex only */

/*
 * Header-only helpers on one shallow octree's bit string t[4] (layout
 * above).  They compile as plain C on the host and, inside a HIP
 * translation unit, as host + device functions.  Nothing is exported from
 * the library for them.
 */
#ifdef __HIP__
#define OC_INLINE static inline __attribute__((host, device))
#else
#define OC_INLINE static inline
#endif

/* Eq. 1: parent of node i >= 1 is floor((i - 1) / 8); the root (i = 0) has
 * none and gets -1. */
OC_INLINE int oc_parent(int i) { return i <= 0 ? -1 : (i - 1) / 8; }

/* Eq. 2: the first child of node i is 8i + 1; its children are
 * 8i + 1 + o for octants o = 0..7. */
OC_INLINE int oc_child(int i) { return 8 * i + 1; }

/* Split bit i (Sec. 3.1: bit j of the 73-bit string, stored LSB first in
 * t[j >> 5]).  Indices outside [0, 73) read 0: the implicit depth-3 voxels
 * are never split. */
OC_INLINE int oc_bit(const uint32_t t[4], int i) {
  if (i < 0 || i >= 73) return 0;
  return (int)((t[i >> 5] >> (i & 31)) & 1u);
}

/* Set bits among indices [0, n), n clamped to [0, 73]. */
OC_INLINE int oc_popc_below(const uint32_t t[4], int n) {
  int c = 0, k;
  if (n > 73) n = 73;
  for (k = 0; n > 0; ++k, n -= 32) {
    const uint32_t w = t[k];
    c += __builtin_popcount(n >= 32 ? w : (w & ((1u << n) - 1u)));
  }
  return c;
}

/* Eq. 3 (the "Data Index" of the supplement): offset of leaf i in its tree's
 * block of rows, counting with popcount.  For i >= 1:
 *   8 * popc(bits [0, pa(i))) + 1 - popc(bits [0, i)) + ((i - 1) mod 8).
 * An unsplit root is the tree's only leaf: oc_data_idx(t, 0) = 0.  The
 * result is meaningful only when node i is a leaf of a canonical tree. */
OC_INLINE int oc_data_idx(const uint32_t t[4], int i) {
  if (i <= 0) return 0;
  return 8 * oc_popc_below(t, (i - 1) / 8) + 1 - oc_popc_below(t, i) + (i - 1) % 8;
}

/* Leaves of a canonical tree: every split adds 7, so 1 + 7 * (set bits). */
OC_INLINE int oc_n_leaves(const uint32_t t[4]) { return 1 + 7 * oc_popc_below(t, 73); }

/* Bit index of the leaf holding local voxel (ld, lh, lw), each in [0, 8)
 * (the voxel addressing of Sec. 3.2: descend from the root while the node
 * is split; at depth k the child's octant takes bit 2 - k of each of d, h,
 * w).  *depth (if not NULL) receives the leaf's depth 0..3; its cell has
 * edge 8 >> depth.  Returns -1 for a voxel outside [0, 8)^3. */
OC_INLINE int oc_leaf_at(const uint32_t t[4], int ld, int lh, int lw, int* depth) {
  int i = 0, d;
  if (ld < 0 || lh < 0 || lw < 0 || ld > 7 || lh > 7 || lw > 7) return -1;
  for (d = 0; d < 3 && oc_bit(t, i); ++d) {
    const int sh = 2 - d;
    i = oc_child(i) + (((ld >> sh) & 1) << 2) + (((lh >> sh) & 1) << 1) + ((lw >> sh) & 1);
  }
  if (depth) *depth = d;
  return i;
}

/* Is the tree canonical (no set bit below an unsplit node, bits 73..127
 * zero)?  1 yes, 0 no. */
OC_INLINE int oc_tree_canonical(const uint32_t t[4]) {
  int i;
  if ((t[2] >> 9) != 0u || t[3] != 0u) return 0;
  for (i = 1; i < 73; ++i)
    if (oc_bit(t, i) && !oc_bit(t, oc_parent(i))) return 0;
  return 1;
}

/* Host check of n_trees trees in host memory: OC_OK if every tree is
 * canonical, OC_ESTRUCT at the first that is not, OC_EINVAL for a null
 * pointer or a negative count.  The device form is oc_validate. */
OC_INLINE int oc_validate_host(const uint32_t* trees_host, int64_t n_trees) {
  int64_t k;
  if (!trees_host || n_trees < 0) return OC_EINVAL;
  for (k = 0; k < n_trees; ++k)
    if (!oc_tree_canonical(trees_host + 4 * k)) return OC_ESTRUCT;
  return OC_OK;
}

/* Static text for a return code. */
const char* oc_error_string(int code);

/* Detail of the last failure on the calling thread ("" if none). */
const char* oc_last_error(void);

/* Library version (major*10000 + minor*100 + patch). */
int oc_version(void);

/* Bytes of workspace needed by oc_build, oc_prefix, oc_validate and the
 * structure calls of pooling/unpooling for n_trees trees. */
size_t oc_structure_workspace(int64_t n_trees);

/*
 * Octree creation from an occupancy grid (Sec. 1: cells that contain data are
 * split recursively down to the finest level).  occ: uint8
 * [n][8gd][8gh][8gw], non-zero = occupied.  Each node at depth 0, 1, 2 whose
 * parent is split is split according to `rule`.  Writes trees and prefix;
 * *n_leaves [host] receives prefix[n_trees].  Synchronizes.
 */
int oc_build(const uint8_t* occ, int n, int gd, int gh, int gw, int rule, uint32_t* trees,
             int64_t* prefix, int64_t* n_leaves, void* ws, size_t ws_bytes, void* stream);

/*
 * oc_build without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid hipMalloc).  Same arguments and results as oc_build; the leaf
 * counts and scan partials go to a static device array inside the library
 * (16.1 MB per device, held until the process ends), so at most 4,194,304
 * trees (e.g. a 512^3 grid in batches of 8); more give OC_EOVERFLOW before
 * any launch.  Calls no allocating routine.  Every call on one device shares
 * that array: calls that may overlap on one device (other streams, other
 * threads) race and must be serialised by the caller.  Synchronizes.
 */
int oc_build_noalloc(const uint8_t* occ, int n, int gd, int gh, int gw, int rule, uint32_t* trees,
                     int64_t* prefix, int64_t* n_leaves, void* stream);

/* prefix from trees: leaves per tree = 1 + 7 * (set bits) (Eq. 3 counted to
 * the end of the tree), exclusive scan over trees.  *n_leaves [host] receives
 * the total.  Synchronizes. */
int oc_prefix(const uint32_t* trees, int64_t n_trees, int64_t* prefix, int64_t* n_leaves,
              void* ws, size_t ws_bytes, void* stream);

/* Counts non-canonical trees into *n_bad [host].  Synchronizes. */
int oc_validate(const uint32_t* trees, int64_t n_trees, int64_t* n_bad, void* ws,
                size_t ws_bytes, void* stream);

/* leaf_info[row] = tree << 10 | bit index of the leaf stored at that row
 * (Eq. 3 inverted).  leaf_info: uint64 [prefix[n_trees]]. */
int oc_leaf_index(const uint32_t* trees, const int64_t* prefix, int64_t n_trees,
                  uint64_t* leaf_info, void* stream);

/* rowmap[n][8gd][8gh][8gw] = row of the leaf holding each voxel (the voxel
 * addressing of Sec. 3.2: tree = voxel/8, local = voxel mod 8, then the
 * smallest cell containing it and Eq. 3).  rowmap: int64. */
int oc_rowmap(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
              int64_t* rowmap, void* stream);

/* Eq. 4: dense[v][k] = data[row of the leaf holding voxel v][k]. */
int oc_oc2ten(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
              const float* data, int c, float* dense, void* stream);

/* Eq. 5: data[leaf][k] = pool over the leaf's voxels of dense[v][k]; pool is
 * OC_POOL_AVG (sum accumulated in double) or OC_POOL_MAX. */
int oc_ten2oc(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
              const float* dense, int c, int pool, float* data, void* stream);

/* Bytes of workspace for oc_conv3x3x3 on a structure with n_trees trees and
 * n_leaves leaves.  *bytes [host].  The size is a bound that holds for every
 * canonical structure of that size and covers every implementation; on the
 * fused MFMA path it is dominated by the per-call boundary sums of split
 * nodes, whose slots it bounds by (n_leaves - n_trees)/7 (every split node
 * adds 7 leaves) at 26*cin*4 + 868 bytes each, in channel blocks by the
 * partial outputs of one input block, n_leaves*cout*4 bytes, and on the GEMM
 * path by one chunk of window sums (about 256 MB). */
int oc_conv3x3x3_workspace(int64_t n_trees, int64_t n_leaves, int cin, int cout, size_t* bytes);

/* Bytes of workspace for oc_conv3x3x3 on this structure: as
 * oc_conv3x3x3_workspace with the boundary-sum slots the structure has (its
 * split trees plus split depth-1 nodes, Sec. 3.1, at least 1) in place of
 * the bound.  The slots are counted on the device: scratch is 256 bytes of
 * device memory (its contents are overwritten), the count runs on stream,
 * and the call synchronizes with it.  *bytes [host].  A workspace of this
 * size serves this structure (and any other with no more slots); the
 * convolution calls take their slot capacity from ws_bytes, so a workspace
 * below the structure's exact size gives wrong results, not an error (one
 * below the one-slot size gives OC_EWORKSPACE). */
int oc_conv3x3x3_workspace_exact(const uint32_t* trees, int n, int gd, int gh, int gw, int64_t n_leaves,
                                 int cin, int cout, size_t* bytes, void* scratch, void* stream);

/* Bytes of workspace for oc_conv3x3x3 on a structure of this size with
 * `slots` boundary-sum slots (split trees plus split depth-1 nodes; values
 * below 1 count as 1, values above the bound as the bound): what
 * oc_conv3x3x3_workspace_exact returns for a structure with that count.
 * Host only.  *bytes [host]. */
int oc_conv3x3x3_workspace_slots(int64_t n_trees, int64_t n_leaves, int cin, int cout, int64_t slots,
                                 size_t* bytes);

/* The boundary-sum slots a workspace of ws_bytes holds for a structure of
 * this size: the convolution calls work with this capacity (the bound at
 * most; 0 where the layer has no fused kernels).  *slots [host]; a
 * workspace below the one-slot size gives OC_EWORKSPACE.  Host only. */
int oc_conv3x3x3_workspace_capacity(int64_t n_trees, int64_t n_leaves, int cin, int cout, size_t ws_bytes,
                                    int64_t* slots);

/*
 * Grid-octree 3x3x3 convolution, Eq. 8 with average pooling: for every leaf,
 * the mean over its cell of the dense convolution of Eq. 7 (zero padding 1,
 * zero outside the grid) applied to oc2ten(in), plus bias, optionally
 * followed by max(0, .).  The output has the input's structure.
 *   in:     float [n_leaves][cin]
 *   weight: float [cout][cin][3][3][3] in Eq. 7's orientation: tap (l,m,n)
 *           multiplies input voxel (i-l+1, j-m+1, k-n+1) for output (i,j,k).
 *   bias:   float [cout] or NULL.
 *   out:    float [n_leaves][cout].
 * Requires n_leaves < 2^31.  ws: at least oc_conv3x3x3_workspace bytes, or
 * the oc_conv3x3x3_workspace_exact bytes of this structure.
 */
int oc_conv3x3x3(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                 int64_t n_leaves, const float* in, int cin, const float* weight,
                 const float* bias, int cout, int relu, float* out, void* ws, size_t ws_bytes,
                 void* stream);

/* As oc_conv3x3x3 with an explicit implementation (OC_CONV_*). */
int oc_conv3x3x3_ex(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                    int64_t n_leaves, const float* in, int cin, const float* weight,
                    const float* bias, int cout, int relu, float* out, void* ws,
                    size_t ws_bytes, int impl, void* stream);

/* The two halves of oc_conv3x3x3_ex, for callers that reuse a structure or
 * time the convolution proper.  prepare writes everything that depends on
 * the structure and the weights into ws (it reads weight, not the features);
 * execute runs the convolution from that workspace and must get the same
 * structure, channel counts and ws as the prepare call before it.  execute
 * also writes per-call scratch into ws (boundary sums of the input,
 * window-sum chunks, channel-block partials) but leaves what prepare wrote
 * intact, so one prepared ws serves any number of executes in stream order;
 * two executes that share one ws and may overlap (different streams) race:
 * give each its own prepared ws. */
int oc_conv3x3x3_prepare(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                         int64_t n_leaves, const float* weight, int cin, int cout, void* ws,
                         size_t ws_bytes, void* stream);
int oc_conv3x3x3_execute(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                         int64_t n_leaves, const float* in, int cin, const float* bias, int cout,
                         int relu, float* out, void* ws, size_t ws_bytes, int impl,
                         void* stream);

/* Does OC_CONV_MFMA support (cin, cout)?  1 yes, 0 no.  Fused variants exist
 * for cin in {4, 8, 16, 32} and cout in [5, 32].  Wider layers with cin a
 * multiple of 32 and cout a multiple of 32 up to 256 (or a fused width below
 * 32) run in channel blocks: Eq. 7 is a sum over input channels, so the
 * layer is computed as (cin/32) x (cout/cb) fused 32 -> cb convolutions; the
 * partial outputs of each input block go to the workspace and are added to
 * the output in block order (after the bias; the ReLU after the last). */
int oc_conv3x3x3_mfma_supported(int cin, int cout);

/*
 * 2x2x2 pooling structure (Eq. 10): input grid 2D x 2H x 2W trees (gd, gh, gw
 * even) -> output D x H x W.  Input trees (2d+a, 2h+b, 2w+c) become octant
 * o = 4a+2b+c of output tree (d,h,w); every input node moves one level down;
 * the output root is always split.  Writes out_trees, out_prefix and
 * *out_n_leaves [host].  Synchronizes.
 */
int oc_pool2_structure(const uint32_t* in_trees, int n, int gd, int gh, int gw,
                       uint32_t* out_trees, int64_t* out_prefix, int64_t* out_n_leaves,
                       void* ws, size_t ws_bytes, void* stream);

/* Eq. 10 data: an output leaf that comes from an input cell of size >= 2
 * copies it; an output unit voxel that comes from a split depth-2 input node
 * takes the maximum of its 8 unit-voxel children.  gd, gh, gw are the input
 * dims; the output structure comes from oc_pool2_structure. */
int oc_pool2_max(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh,
                 int gw, const float* in, int c, const uint32_t* out_trees,
                 const int64_t* out_prefix, float* out, void* stream);

/*
 * 2x2x2 unpooling structure.  guide_trees == NULL: plain unpooling (Eq. 12):
 * input tree (d,h,w) spawns output trees (2d+a, 2h+b, 2w+c); input node 1+o
 * becomes the root of output tree o = 4a+2b+c and every node below it moves
 * one level up; an unsplit input root spawns 8 unsplit trees.
 * guide_trees != NULL: guided unpooling (the remark after Eq. 12): the output
 * structure is the guide (2gd x 2gh x 2gw trees), which must pool to the
 * input structure (else OC_ESTRUCT).  gd, gh, gw are the input dims.  Writes
 * out_trees, out_prefix and *out_n_leaves [host].  Synchronizes.
 */
int oc_unpool2_structure(const uint32_t* in_trees, int n, int gd, int gh, int gw,
                         const uint32_t* guide_trees, uint32_t* out_trees, int64_t* out_prefix,
                         int64_t* out_n_leaves, void* ws, size_t ws_bytes, void* stream);

/* Eq. 12 data: every output leaf copies the input leaf that holds its voxels
 * at half resolution (plain or guided structure alike).  gd, gh, gw are the
 * input dims; out_trees/out_prefix come from oc_unpool2_structure. */
int oc_unpool2(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh, int gw,
               const float* in, int c, const uint32_t* out_trees, const int64_t* out_prefix,
               float* out, void* stream);

/* Pointwise max(0, x) on leaf data (pointwise ops act on leaf data alone,
 * Sec. 3.2).  In place allowed. */
int oc_relu(float* data, int64_t count, void* stream);

/*
 * Gradients.  Each takes the output gradient (dout, laid out as the forward
 * output) and writes gradients laid out as the forward operands; the caller
 * owns every buffer, and outputs must not alias inputs except in
 * oc_relu_backward.  They follow from the forward definitions by the chain
 * rule (back-propagation through the layers of Sec. 3, trained end to end as
 * in Sec. 5).
 */

/* Bytes of workspace for oc_conv3x3x3_backward.  *bytes [host]. */
int oc_conv3x3x3_backward_workspace(int64_t n_trees, int64_t n_leaves, int cin, int cout,
                                    size_t* bytes);

/*
 * Gradient of oc_conv3x3x3 (Eq. 8 with average pooling) without its ReLU:
 * apply oc_relu_backward to dout first when the forward call fused one.
 *   dout:    float [n_leaves][cout], the gradient of the convolution output.
 *   din:     float [n_leaves][cin] or NULL: the input gradient.  With
 *            g_l = dout_l / |l| spread over the voxels of output leaf l, input
 *            leaf l' receives |l'| times the convolution of g with the
 *            flipped, channel-transposed kernel (the adjoint of Eq. 7 summed
 *            over the cell).  Needs weight.
 *   dweight: float [cout][cin][3][3][3] or NULL (overwritten, not
 *            accumulated): sum over leaves of g_l times the window sums of
 *            the forward input.  Needs in.
 *   dbias:   float [cout] or NULL: the column sums of dout.
 * cin, cout in [1, 256]; n_leaves < 2^31.  ws: at least
 * oc_conv3x3x3_backward_workspace bytes.  Deterministic: the sums run in a
 * fixed order.
 */
int oc_conv3x3x3_backward(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh,
                          int gw, int64_t n_leaves, const float* in, int cin, const float* weight,
                          int cout, const float* dout, float* din, float* dweight, float* dbias,
                          void* ws, size_t ws_bytes, void* stream);

/* Gradient of oc_pool2_max (Eq. 10).  Arguments as oc_pool2_max; in is the
 * forward input, dout [out leaves][c], din [in leaves][c] (every row
 * written).  An output leaf that copies an input leaf passes its gradient
 * through; one that takes the maximum of 8 unit voxels passes it, channel by
 * channel, to the first of them (in child order) holding the maximum. */
int oc_pool2_max_backward(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh,
                          int gw, const float* in, int c, const uint32_t* out_trees,
                          const int64_t* out_prefix, const float* dout, float* din, void* stream);

/* Gradient of oc_unpool2 (Eq. 12, plain or guided).  Arguments as
 * oc_unpool2, plus in_n_leaves, the row count of din [in_n_leaves][c]: every
 * input leaf receives the sum of dout over the output leaves that copy it
 * (in output row order). */
int oc_unpool2_backward(const uint32_t* in_trees, const int64_t* in_prefix, int n, int gd, int gh,
                        int gw, int64_t in_n_leaves, int c, const uint32_t* out_trees,
                        const int64_t* out_prefix, const float* dout, float* din, void* stream);

/* Gradient of oc_relu given its output: din = dout where out > 0, else 0.
 * din may alias dout; count 0 does nothing (the pointers may then be NULL). */
int oc_relu_backward(const float* out, const float* dout, float* din, int64_t count, void* stream);

/*
 * Channel concatenation of two leaf arrays on one structure: out[row] =
 * [a[row] (ca channels), b[row] (cb channels)], the skip connections of the
 * encoder-decoder network (Sec. 5 and the segmentation architecture table:
 * concat of an encoder output and the unpooled decoder features at the
 * same resolution, i.e. on the same structure).
 *   a: float [n_rows][ca], b: float [n_rows][cb], out: float [n_rows][ca+cb].
 * n_rows 0 does nothing (pointers may then be NULL).
 */
int oc_concat(const float* a, int ca, const float* b, int cb, int64_t n_rows, float* out,
              void* stream);

/* Gradient of oc_concat: da[row] = dout[row][0..ca), db[row] = dout[row][ca..ca+cb).
 * da or db may be NULL (that part is not written). */
int oc_concat_backward(const float* dout, int ca, int cb, int64_t n_rows, float* da, float* db,
                       void* stream);

/* out = a + b elementwise on leaf data (pointwise, Sec. 3.2): the gradient
 * of a layer output that feeds two layers (an encoder output used by the
 * next level and by a concat) is the sum of both.  out may alias a or b
 * (entirely, not in part); count 0 does nothing. */
int oc_add(const float* a, const float* b, float* out, int64_t count, void* stream);

/*
 * Point clouds (Sec. 5, the facade segmentation input: the points are mapped
 * into the grid-octree; a leaf holding points takes the mean of their
 * features and the majority of their labels).
 *   pts:   float [n_pts][3], coordinates in voxels along (d, h, w) of the
 *          8gd x 8gh x 8gw grid; a point lies in voxel floor(coordinate).
 *   batch: int32 [n_pts], the sample of each point, or NULL (all sample 0).
 * Points outside the grid (or of a sample outside [0, n)) are ignored.
 */

/* occ [n][8gd][8gh][8gw] (uint8): 1 where a point lies, else 0 (cleared by
 * the call).  Build the structure from occ with oc_build. */
int oc_points_voxelize(const float* pts, const int32_t* batch, int64_t n_pts, int n, int gd, int gh,
                       int gw, uint8_t* occ, void* stream);

/* rows [n_pts] (int32): the row of the leaf holding each point (Eq. 3 on the
 * bit index of its cell), -1 for an ignored point.  Requires n_leaves < 2^31. */
int oc_points_leaf_rows(const uint32_t* trees, const int64_t* prefix, int n, int gd, int gh, int gw,
                        const float* pts, const int32_t* batch, int64_t n_pts, int32_t* rows,
                        void* stream);

/* Bytes of scratch for oc_points_average (n_labels = 1) and oc_points_vote. */
size_t oc_points_workspace(int64_t n_leaves, int n_labels);

/* out [n_leaves][c + 1]: channel 0 = 1 where at least one point fell into the
 * leaf, else 0 (the binary occupancy feature); channels 1..c = the mean of
 * the points' features feat [n_pts][c] (0 without points).  The sums run in
 * atomic order, so the means may differ in the last bits between runs. */
int oc_points_average(const int32_t* rows, int64_t n_pts, const float* feat, int c, int64_t n_leaves,
                      float* out, void* ws, size_t ws_bytes, void* stream);

/* out [n_leaves] (int32): the most frequent label in [0, n_labels) among the
 * leaf's points, the smallest of tied labels, -1 without labelled points.
 * Exact (integer counts). */
int oc_points_vote(const int32_t* rows, int64_t n_pts, const int32_t* labels, int n_labels,
                   int64_t n_leaves, int32_t* out, void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OCTNET_HIP_H */
