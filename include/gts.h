/*
 * gts.h -- C ABI of libgts: exact path-based TreeShap for AMD Instinct MI355X
 * (gfx950), after Mitchell, Frank & Holmes, "GPUTreeShap: Massively Parallel
 * Exact Calculation of SHAP Scores for Tree Ensembles" (arXiv 2010.13972).
 *
 * Pipeline (Section 3, steps 1-4):
 *   gts_extract_paths   host   ensemble -> merged unique root-to-leaf paths
 *   gts_extract_paths_device  the same on the GPU, bit for bit
 *   gts_extract_paths_device_noalloc  the same without a caller workspace
 *   gts_pack_paths      host   paths -> bins of <= 64 path elements
 *   gts_model_layout    host   packed paths -> one device-ready byte blob
 *   gts_prepare_model   host   the three steps above in one pass
 *   gts_plan_model      host   the same without writing the paths: counts,
 *                              packing and each path's place, for
 *   gts_build_model_device  device  which writes the same blob on the GPU
 *   gts_shap            device SHAP values              phi[rows][G][M+1]
 *   gts_shap_interactions device SHAP interaction values phi[rows][G][M+1][M+1]
 *   gts_launch_config   host   the launch shape the two calls above choose
 *   gts_prune_model     device a copy of a model without the paths that no
 *                              row of one batch reaches, for the two device
 *                              calls above on that batch
 *
 * Conventions shared by every call:
 *   - All memory is owned by the caller.  The library calls no device
 *     allocator and never frees caller memory; its only device memory of its
 *     own is the fixed workspace array of gts_extract_paths_device_noalloc.
 *     No result depends on an earlier call; the host calls reuse a pool of
 *     worker threads (up to 16 and the process's cores; two fewer for calls
 *     under 128 k nodes when it has 8 or more; started on first use) and
 *     gts_prepare_model reuses per-thread working memory.  Calls from several
 *     threads may run at once (gts_set_host_threads).
 *   - Every call returns a gts_status; on failure gts_last_error() returns a
 *     message for the calling thread (valid until that thread's next call).
 *   - A split sends x to the left child iff x < threshold; a path element
 *     holds the half-open range [lower, upper) (Section 3.1).
 *   - Feature values must be finite.  A NaN makes every range test false
 *     (the element-wise test of the paper's kernel listing), which is not the
 *     tree's own routing; missing values are not supported.
 *   - M = number of features, G = number of output groups (classes).
 */
#ifndef GTS_H
#define GTS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gts_status {
  GTS_OK = 0,
  GTS_EINVAL = 1,    /* bad argument or malformed ensemble / layout */
  GTS_EPATHLEN = 2,  /* a merged path is longer than the bin capacity (<= 64) */
  GTS_EBUFSIZE = 3,  /* output capacity too small; required sizes were written */
  GTS_ENOMEM = 4,    /* host allocation failed */
  GTS_EDEVICE = 5    /* a HIP call or kernel launch failed */
} gts_status;

typedef enum gts_dtype { GTS_F32 = 0, GTS_F64 = 1 } gts_dtype;

/* Bin-packing heuristics of Section 3.3 / Table 1. */
typedef enum gts_pack_alg {
  GTS_PACK_BFD = 0,  /* Best-Fit-Decreasing (the paper's choice, Section 4.1) */
  GTS_PACK_FFD = 1,  /* First-Fit-Decreasing */
  GTS_PACK_NF = 2,   /* Next-Fit, paths in their input order */
  GTS_PACK_NONE = 3  /* one path per bin (the "none" baseline of Table 5) */
} gts_pack_alg;

/*
 * A tree ensemble as flat node lists: per node the lists {v, a, b, t, r, d}
 * of Section 2.1 (leaf value, left child, right child, threshold, cover,
 * feature).  Tree k owns nodes [tree_node_offsets[k], tree_node_offsets[k+1]);
 * child indices are local to the tree, the root is local index 0, and a leaf
 * has left == right == -1.  feature/threshold are ignored on leaves, value on
 * internal nodes.  cover must be finite and >= 0; a ratio with a zero-cover
 * parent is taken as 0.  tree_group[k] in [0, G) is the output the tree adds
 * to.  All pointers are host pointers.
 */
typedef struct gts_ensemble {
  int32_t num_features;              /* M >= 1 */
  int32_t num_groups;                /* G >= 1 */
  int64_t num_trees;                 /* T >= 0 */
  int64_t num_nodes;                 /* tree_node_offsets[T] */
  const int64_t *tree_node_offsets;  /* [T+1], non-decreasing, starts at 0 */
  const int32_t *tree_group;         /* [T] */
  const int32_t *left;               /* [num_nodes] */
  const int32_t *right;              /* [num_nodes] */
  const int32_t *feature;            /* [num_nodes] */
  const float *threshold;            /* [num_nodes] */
  const double *cover;               /* [num_nodes] */
  const double *value;               /* [num_nodes] */
} gts_ensemble;

/*
 * One element of a unique path: the fields of the paper's PathElement
 * (Listing 1) plus the output group of the path's tree.  The first element of
 * every path is its root (feature_idx -1, range (-inf, +inf), zero_fraction 1);
 * v is the path's leaf value on every element.  40 bytes, naturally aligned.
 */
typedef struct gts_path_element {
  int64_t path_idx;       /* unique path index */
  int32_t feature_idx;    /* split feature, -1 for the root element */
  int32_t group;          /* output group of the path's tree */
  float lower;            /* feature range [lower, upper) */
  float upper;
  double zero_fraction;   /* product of cover ratios along the path */
  double v;               /* leaf value at the end of the path */
} gts_path_element;

/*
 * Device-ready model produced by gts_model_layout.  The fields describe the
 * byte blob the caller copies to the device; treat them as read-only.
 */
#define GTS_MODEL_SORTED_BINS 1
#define GTS_MODEL_PRUNED 2

typedef struct gts_model {
  uint32_t magic;
  int32_t dtype;           /* gts_dtype of zero fractions, leaf values, phi */
  int32_t num_features;    /* M */
  int32_t num_groups;      /* G */
  int32_t max_path_len;    /* longest path, root included */
  int32_t flags;           /* GTS_MODEL_SORTED_BINS: inside every bin, paths
                              are in non-increasing length order (BFD, FFD);
                              GTS_MODEL_PRUNED: from gts_prune_model, whose
                              counts below are capacities */
  int64_t num_elements;
  int64_t num_paths;
  int64_t num_bins;
  int64_t bytes;           /* size of the blob */
  int64_t off[16];         /* byte offsets of the blob's arrays */
} gts_model;

/*
 * gts_extract_paths -- Sections 3.1 and 3.2 (extract paths, remove duplicate
 * features).
 *
 * Walks every tree (trees in input order, leaves in depth-first preorder with
 * the left child first) and emits one path per leaf: its root element, then
 * one element per distinct split feature in ascending feature order.  A left
 * turn at threshold t bounds the range above by t, a right turn below by t;
 * repeated features intersect their ranges and multiply their zero fractions
 * (child cover / parent cover) in root-to-leaf order.
 *
 * out       host array of `capacity` elements, or NULL to query sizes only.
 * num_elements, num_paths  (out) totals; always written on GTS_OK and
 *           GTS_EBUFSIZE.
 * bias      (out, may be NULL) host double[G]: per group the sum over its
 *           paths of v times the product of the path's zero fractions -- the
 *           expected model output f of the empty feature set (the bias term
 *           phi_0 of Eq. 1).  Each tree sums its paths' terms in path order,
 *           then each group sums its trees' sums in tree order.
 * Errors: GTS_EINVAL for out-of-range children, a node reached twice (cycle
 * or shared child), feature outside [0, M), group outside [0, G), negative or
 * non-finite cover, NaN threshold; GTS_EBUFSIZE if capacity is too small.
 */
gts_status gts_extract_paths(const gts_ensemble *ens, gts_path_element *out,
                             int64_t capacity, int64_t *num_elements,
                             int64_t *num_paths, double *bias);

/*
 * gts_extract_workspace_bytes -- size of the device workspace that
 * gts_extract_paths_device needs for an ensemble of num_trees trees and
 * num_nodes nodes (about 52 bytes per node).  Errors: GTS_EINVAL for NULL
 * bytes or negative sizes.
 */
gts_status gts_extract_workspace_bytes(int64_t num_trees, int64_t num_nodes, int64_t *bytes);

/*
 * gts_extract_paths_device -- Sections 3.1 and 3.2 on the GPU: the output of
 * gts_extract_paths (same elements in the same order, bit for bit, and the
 * same bias), from an ensemble whose node arrays are in device memory.  One
 * thread per leaf walks up to its root; scans over trees and paths place the
 * paths; each tree sums its paths' bias terms in path order, each group its
 * trees in tree order (the host's order).
 *
 * ens       host struct; num_features, num_groups, num_trees, num_nodes are
 *           host values, every array pointer is a DEVICE pointer (same
 *           layout as for gts_extract_paths).
 * d_out     device array of `capacity` elements, or NULL to compute sizes
 *           only.
 * num_elements, num_paths  (out, host) totals; written on GTS_OK and
 *           GTS_EBUFSIZE.
 * d_bias    device double[G] or NULL.
 * d_workspace  caller's device memory of workspace_bytes >=
 *           gts_extract_workspace_bytes(num_trees, num_nodes); its contents
 *           are overwritten and may be reused once the stream has passed the
 *           call's work.
 * stream    hipStream_t (NULL = default stream).  The call waits for the
 *           stream twice (to read the path and element counts); the writes of
 *           d_out and d_bias are enqueued and complete with the stream.
 * Errors: GTS_EINVAL for a malformed ensemble.  Unlike the host call, which
 * checks only the nodes reachable from each root, every node is checked
 * (cover, child indices, feature, threshold, leaf value, at most one parent,
 * no parent for a root); leaves not reachable from their root are skipped,
 * as on the host.  Paths deeper than 256 splits give GTS_EINVAL, merged
 * paths of more than 63 features GTS_EPATHLEN (a bin holds at most 64
 * elements); GTS_EBUFSIZE for a workspace or capacity too small;
 * GTS_EDEVICE if a HIP call fails.
 */
gts_status gts_extract_paths_device(const gts_ensemble *ens, gts_path_element *d_out,
                                    int64_t capacity, int64_t *num_elements,
                                    int64_t *num_paths, double *d_bias, void *d_workspace,
                                    int64_t workspace_bytes, void *stream);

/*
 * gts_extract_paths_device_noalloc -- gts_extract_paths_device for callers
 * that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation).  Same arguments, output,
 * order and errors as gts_extract_paths_device, without d_workspace: the
 * workspace is a fixed array of GTS_EXTRACT_NOALLOC_BYTES bytes in the
 * library's device code, one per device, held from module load until the
 * process ends.  The call itself allocates nothing (no hipMalloc, no
 * allocating library routine).
 *
 * Limit: an ensemble whose workspace (gts_extract_workspace_bytes) exceeds
 * GTS_EXTRACT_NOALLOC_BYTES (64 MiB, about 1.2 million nodes) gets GTS_EINVAL
 * before any device work.  Every call on a device shares that device's array
 * and leaves its contents behind (each call initialises what it reads):
 * calls that overlap on one device -- on different streams or from different
 * threads -- race and are not supported; serialise them.
 */
#define GTS_EXTRACT_NOALLOC_BYTES (64LL << 20)

gts_status gts_extract_paths_device_noalloc(const gts_ensemble *ens, gts_path_element *d_out,
                                            int64_t capacity, int64_t *num_elements,
                                            int64_t *num_paths, double *d_bias, void *stream);

/*
 * gts_pack_paths -- Section 3.3 (bin packing for work allocation).
 *
 * Items are paths (contiguous runs starting at a root element, as produced by
 * gts_extract_paths) of size = path length; bins hold `bin_capacity` lanes
 * (<= 64, one lane per path element on a wave64).  Each output group is packed
 * on its own, groups ascending, bins numbered in opening order.
 *   BFD: items by non-increasing size (ties: lower path position first); each
 *        goes to the feasible bin with the smallest residual (ties: lower bin).
 *   FFD: same order; the lowest-numbered feasible bin.
 *   NF:  input order; the current bin if it fits, else a new bin.
 *   NONE: one path per bin, input order.
 * A bin may be filled exactly to capacity.  Within a bin, paths are laid out
 * in placement order.
 *
 * packed       host array [num_elements]: the elements regrouped bin by bin.
 * bin_offsets  host array [offsets_capacity]; receives num_bins+1 element
 *              offsets into `packed`.  May be NULL with offsets_capacity 0 to
 *              query num_bins (packed is then not written).
 * Errors: GTS_EPATHLEN if a path is longer than bin_capacity;
 * GTS_EINVAL for capacity outside [1, 64], an unknown alg, or input that is
 * not a sequence of rooted paths; GTS_EBUFSIZE when offsets_capacity <
 * num_bins + 1 (num_bins is written).
 */
gts_status gts_pack_paths(const gts_path_element *elems, int64_t num_elements,
                          int32_t bin_capacity, int32_t alg,
                          gts_path_element *packed, int64_t *bin_offsets,
                          int64_t offsets_capacity, int64_t *num_bins);

/*
 * gts_model_layout -- marshal packed paths into the blob the device kernels
 * read (structure-of-arrays, every array 256-byte aligned).
 *
 * packed, bin_offsets, num_bins: the output of gts_pack_paths (bins must not
 *           mix groups).  bias: host double[G] from gts_extract_paths.
 * dtype     GTS_F32 or GTS_F64: precision of zero fractions, leaf values and
 *           of the whole SHAP recurrence and accumulation.
 * model     (out) descriptor; model->bytes is the blob size.
 * host_blob host buffer of blob_capacity bytes, or NULL to size only (the
 *           input is then only counted; it is validated when the blob is
 *           written).
 * Errors: GTS_EINVAL for inconsistent input, GTS_EPATHLEN for a path longer
 * than 64, GTS_EBUFSIZE if blob_capacity < model->bytes.
 */
gts_status gts_model_layout(const gts_path_element *packed, int64_t num_elements,
                            const int64_t *bin_offsets, int64_t num_bins,
                            int32_t num_features, int32_t num_groups,
                            const double *bias, int32_t dtype, gts_model *model,
                            void *host_blob, int64_t blob_capacity);

/*
 * gts_prepare_model -- Sections 3.1-3.3 in one host pass: extract and merge
 * the paths of `ens`, pack them (bin_capacity, alg as gts_pack_paths) and
 * write the device blob, without building the intermediate
 * gts_path_element arrays; trees are walked, sorted and written on several
 * host threads.  The blob and descriptor are byte for byte those of
 * gts_model_layout(gts_pack_paths(gts_extract_paths(ens))).  Its working
 * memory (about 35 bytes per path element) stays with the calling thread and
 * is reused by that thread's next call.
 *
 * host_blob host buffer of blob_capacity bytes, or NULL to size only (then
 *           model->bytes gives the size).  bias (out, may be NULL) double[G].
 * Errors: as gts_extract_paths for a malformed ensemble; GTS_EPATHLEN if a
 * merged path is longer than bin_capacity; GTS_EBUFSIZE if blob_capacity <
 * model->bytes (model is written).
 */
gts_status gts_prepare_model(const gts_ensemble *ens, int32_t bin_capacity, int32_t alg,
                             int32_t dtype, gts_model *model, void *host_blob,
                             int64_t blob_capacity, double *bias);

/*
 * gts_plan_model -- gts_prepare_model split between host and device: on the
 * host, the walk that validates the trees and counts every path's merged
 * features (Sections 3.1-3.2), the packing (Section 3.3) and each path's
 * place in the blob; gts_build_model_device then extracts and merges the
 * paths on the GPU, writes them to those places and sums the bias.  The blob
 * it writes is byte for byte the one gts_prepare_model writes for the same
 * ensemble, bin capacity, algorithm and dtype.  Only for models whose every
 * launch runs one path per wave (M <= 17 in fp32, M <= 11 in fp64), where a
 * path's element order depends on nothing but the path.
 *
 * model      out: the descriptor of the blob gts_build_model_device writes.
 * plan       out: counts, the plan blob's size and its arrays' byte offsets:
 *            off[0] uint64 path_dirs[P] path p's turns from its tree's root:
 *                                       bit k set when its k-th split sends
 *                                       it right (paths of at most 64 splits)
 *            off[1] int32 path_dest[P]  element offset of path p's root in
 *                                       the model blob
 *            off[2] int32 tree_paths[T+1]  first path of every tree
 *            off[3] int32 bin_start[K+1]   as in the model blob
 *            off[4] int32 group_bins[G+1]  as in the model blob
 * host_plan  host memory of `capacity` bytes for the plan blob, or NULL for
 *            the descriptors only.
 * Errors: as gts_prepare_model; GTS_EINVAL for a model with more features
 * than above, a path of more than 64 splits, or 2^31 nodes or paths or more;
 * GTS_EBUFSIZE if capacity is smaller than plan->bytes.
 */
typedef struct gts_plan {
  int64_t num_paths;   /* P */
  int64_t num_trees;   /* T */
  int64_t num_bins;    /* K */
  int64_t num_nodes;   /* of the ensemble the plan was made for */
  int64_t bytes;       /* size of the plan blob */
  int64_t off[5];
} gts_plan;

gts_status gts_plan_model(const gts_ensemble *ens, int32_t bin_capacity, int32_t alg,
                          int32_t dtype, gts_model *model, gts_plan *plan, void *host_plan,
                          int64_t capacity);

/*
 * gts_build_workspace_bytes -- device workspace gts_build_model_device needs
 * for this plan: 8 bytes per path and per tree.
 */
gts_status gts_build_workspace_bytes(const gts_plan *plan, int64_t *bytes);

/*
 * gts_build_model_device -- the model blob of a plan, written on the GPU
 * (Sections 3.1-3.2 for the elements): one thread per path follows its
 * turns from its tree's root down to its leaf, merging as it goes (ranges
 * intersected, zero fractions multiplied in root-to-leaf order, features
 * ascending), and writes the root and the elements, the zero-fraction ones
 * first, at the path's place; each tree sums its paths' bias terms
 * v * prod(z) in path order and each group its trees' sums in tree order,
 * as on the host.  The result equals gts_prepare_model's blob byte for byte.
 *
 * ens        host struct whose array pointers are DEVICE pointers (as for
 *            gts_extract_paths_device), holding the ensemble the plan was made
 *            from; it is not validated again.
 * model, plan  descriptors from gts_plan_model.
 * d_plan     device copy of the plan blob.
 * d_model    device memory of model->bytes, overwritten.
 * d_workspace  device memory of gts_build_workspace_bytes, overwritten; free
 *            for reuse once the stream has passed the call's work.
 * stream     hipStream_t; the work is only enqueued (no waits).
 * Errors: GTS_EINVAL for NULL pointers, a descriptor not from
 * gts_model_layout or gts_plan_model, or an ensemble whose counts differ
 * from the plan's; GTS_EBUFSIZE for a workspace too small; GTS_EDEVICE if
 * a launch fails.
 */
gts_status gts_build_model_device(const gts_ensemble *ens, const gts_model *model,
                                  const gts_plan *plan, const void *d_plan, void *d_model,
                                  void *d_workspace, int64_t workspace_bytes, void *stream);

/*
 * gts_shap -- SHAP values, Eq. (2), by the per-path permutation-weight
 * recurrence of Algorithm 1 (EXTEND over a path's elements, then UNWIND of
 * each element and a sum), evaluated per (row, path) over the packed bins
 * of Section 3.4.  A (row, path) with an element of zero fraction whose range
 * misses the row contributes exactly nothing (Algorithm 1 prunes such
 * subtrees) and may be skipped.  The kernels for paths longer than 16
 * features use per-lane private memory that the HIP runtime provides with
 * the launch; the others use none of their own beyond LDS and, at the
 * tightest register caps, a few words of register spills.
 *
 * model    host descriptor from gts_model_layout.
 * d_model  device copy of the blob.
 * d_X      device float[rows][ld_x], row-major, ld_x >= M.
 * d_phi    device array [rows][G][M+1] of the model dtype.  Overwritten:
 *          phi[r][g][i] for i < M is feature i's SHAP value for output g;
 *          phi[r][g][M] is the bias.
 * stream   hipStream_t (NULL = default stream).  The call only enqueues work
 *          and returns; results are ready when the stream reaches them.
 * rows == 0 is a no-op.  Errors: GTS_EINVAL for NULL pointers, a descriptor
 * that is not from gts_model_layout, rows < 0, ld_x < M, or an M whose phi
 * and X rows do not fit in a workgroup's LDS at 4 rows per tile (on a
 * 160 KB-LDS device: M <= 4567 in fp32, M <= 2852 in fp64; for
 * gts_shap_interactions M <= 132 in fp32, M <= 90 in fp64), checked before
 * any launch; GTS_EDEVICE if a launch fails.
 */
gts_status gts_shap(const gts_model *model, const void *d_model,
                    const float *d_X, int64_t rows, int64_t ld_x, void *d_phi,
                    void *stream);

/*
 * gts_shap_interactions -- SHAP interaction values, Eq. (3)-(6), computed per
 * path by conditioning on each of its features in turn (Sections 2.2 and
 * 3.5): only features on a path interact through it.
 *
 * d_phi    device array [rows][G][M+1][M+1] of the model dtype, overwritten:
 *          [i][j] (i != j < M) the interaction of features i and j, [i][i]
 *          from Eq. (6), [M][M] the bias, the rest of row and column M zero.
 * Other arguments and errors as gts_shap.
 */
gts_status gts_shap_interactions(const gts_model *model, const void *d_model,
                                 const float *d_X, int64_t rows, int64_t ld_x,
                                 void *d_phi, void *stream);

/*
 * gts_launch_config -- the launch that gts_shap (interactions == 0) or
 * gts_shap_interactions (interactions != 0) makes for this model and row
 * count on the calling thread's current device, without launching anything.
 * For tuning and tests.  The decomposition it reports is the work split of
 * Sections 3.3-3.4: bins of paths as work units, a tile of rows per
 * workgroup.
 *
 * rows_per_tile  rows of a workgroup's phi tile (64, 32, 16, 8 or 4); below
 *                64, a wave runs 64 / rows_per_tile paths at once
 * waves          waves (64 lanes) per workgroup
 * private_tiles  1 if every wave has a phi tile of its own (no LDS atomics)
 * slices         bin slices per (row tile, output group); above 1 the
 *                slices add their tiles to phi atomically after a clearing
 *                pass
 * workgroups     grid size (0 for rows == 0)
 * lds_bytes      LDS per workgroup
 * Errors: GTS_EINVAL as gts_shap, for out == NULL, or when a phi row does
 * not fit in a workgroup's LDS; GTS_EDEVICE without a HIP device.
 */
typedef struct gts_launch {
  int32_t rows_per_tile;
  int32_t waves;
  int32_t private_tiles;
  int32_t slices;
  int64_t workgroups;
  int64_t lds_bytes;
} gts_launch;

gts_status gts_launch_config(const gts_model *model, int64_t rows, int32_t interactions,
                             gts_launch *out);

/*
 * gts_prune_workspace_bytes -- device workspace (bytes) that gts_prune_model
 * needs for this model and row count on the calling thread's current device:
 * about 16 bytes per path element for fp32 models (20 for fp64) plus 4 bytes
 * per feature per row.  Errors: GTS_EINVAL as gts_prune_model.
 */
gts_status gts_prune_workspace_bytes(const gts_model *model, int64_t rows, int64_t *bytes);

/*
 * gts_prune_model -- the model without the paths that contribute nothing to
 * any row of one batch.  A (row, path) pair whose path has an element of zero
 * fraction with a range that misses the row's value contributes exactly
 * nothing to that row's SHAP and interaction values (Algorithm 1 prunes such
 * zero-cover subtrees).  A path is dropped when one of its zero-fraction
 * elements has a range [lower, upper) that holds the value of no row of d_X
 * (the same range test as the kernels', on the same keys); every other path
 * is kept, with its elements unchanged.  gts_shap and gts_shap_interactions
 * on the pruned model and the same rows give the values they give on the
 * model itself, up to the rounding of a different summation order: the kept
 * paths are rebinned by output group and length (longest first), each bin
 * holding paths of one length (64 / length of them; the last bin of a length
 * fewer).  The bias is the model's.
 *
 * model        host descriptor from gts_model_layout (not from this call).
 * d_model      device copy of its blob.
 * d_X, rows, ld_x  the batch, as for gts_shap (rows == 0: nothing is
 *              launched and the pruned model must not be used).
 * d_workspace  device memory of gts_prune_workspace_bytes bytes, aligned to
 *              256 bytes, owned by the caller; it holds the pruned blob, so
 *              it must stay untouched while the pruned model is in use.
 * pruned       out: the pruned model's host descriptor, written before the
 *              call returns.  Its num_elements, num_paths and num_bins are
 *              capacities (the model's own counts; the device holds the
 *              pruned counts) and GTS_MODEL_PRUNED and GTS_MODEL_SORTED_BINS
 *              are set.  Valid only for the rows of d_X: other rows may reach
 *              dropped paths.
 * d_pruned     out: device address of the pruned blob, inside d_workspace.
 * stream       hipStream_t; the work is enqueued (five launches) and the
 *              pruned blob is complete when the stream reaches its end, so
 *              later calls on the same stream may use it.
 * Errors: GTS_EINVAL for NULL pointers, a descriptor not from
 * gts_model_layout or one from this call, rows < 0, ld_x < M, a misaligned
 * workspace, or a model with 2^31 elements or more; GTS_EBUFSIZE if
 * workspace_bytes is too small; GTS_EDEVICE if a launch fails.
 */
gts_status gts_prune_model(const gts_model *model, const void *d_model, const float *d_X,
                           int64_t rows, int64_t ld_x, void *d_workspace,
                           int64_t workspace_bytes, gts_model *pruned, void **d_pruned,
                           void *stream);

/*
 * gts_set_host_threads -- caps the host threads (the caller included) that
 * the host calls made from the calling thread use: the tree walks and blob
 * writing of gts_extract_paths, gts_pack_paths, gts_model_layout and
 * gts_prepare_model.  n = 0 restores the default (every core of the
 * process's affinity mask, up to 16).  The setting belongs to the calling
 * thread and lasts until its next call.  For running several preparations
 * at once, each on part of the cores (a pipeline that prepares the models
 * of its next steps in parallel): calls from different threads share one
 * pool of workers, and a free worker serves the preparation that started
 * first, so the oldest call in flight finishes soonest.  Results never
 * depend on the thread count.
 * Errors: GTS_EINVAL for n < 0.
 */
gts_status gts_set_host_threads(int32_t n);

/* Message describing the calling thread's most recent failure ("" if none). */
const char *gts_last_error(void);

/* Library version string. */
const char *gts_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GTS_H */
