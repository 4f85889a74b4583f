/*
 * sb.h -- C ABI of libsketchboost: sketched multioutput split search on one
 * AMD Instinct MI355X (gfx950).
 *
 * The library implements the split-search hot path of SketchBoost (Iosipoi &
 * Vakhrushev, "SketchBoost: Fast Gradient Boosted Decision Tree for
 * Multioutput Problems", NeurIPS 2022, arXiv 2211.12858):
 *
 *   sketch the n x d gradient matrix G to k columns (Section 3.1 Top Outputs,
 *   Section 3.2 Random Sampling, Section 3.3 Random Projections) -> per node,
 *   feature and bin histograms of the k sketch columns plus the hessian
 *   column (Section 3.4, histogram algorithm) -> score every threshold with
 *   S(R) = sum_t (sum_{i in R} g_it)^2 / (sum_{i in R} h_i + lambda)
 *   (Section 2, eq. 4, in the hessian-free form S_G of Section 3) -> best
 *   split per node -> partition the node's rows; repeated level by level
 *   (depth-wise growth, Appendix B.1).
 *
 * Conventions shared by every call
 * --------------------------------
 * - All array arguments are DEVICE pointers owned by the caller (for example
 *   torch tensors).  The library never allocates or frees device memory;
 *   scratch memory is passed in as `ws` / `ws_bytes`, sized by
 *   sb_workspace_bytes().  `ws` must be 256-byte aligned.
 * - Every call checks its scalar arguments and pointer presence on the host
 *   first; on failure it returns SB_E_ARG / SB_E_SHAPE / SB_E_UNSUPPORTED
 *   before touching the device, and sb_last_error() explains why.  Then it
 *   enqueues kernels on `stream` (a hipStream_t; NULL = default stream) and
 *   returns without waiting.  Outputs are valid once the stream has reached
 *   that point.  A launch failure returns SB_E_DEVICE.
 * - Device-resident index arguments (row indices, node offsets, build lists,
 *   split features) are clamped into range by the kernels so that a bad
 *   value can never make an access leave its buffer; results for such input
 *   are unspecified.  Floating-point inputs must be finite.
 * - Node numbering is level-local: node j of a level has children 2j (rows
 *   with bin <= threshold, "left") and 2j+1 ("right") on the next level.
 * - Calls on different streams may run concurrently if their workspaces and
 *   outputs do not overlap.  Only the error text is per-thread state.
 * - Sizes: n < 2^31 rows, m <= 65535 features, 2 <= n_bins <= 256,
 *   1 <= k <= 255 sketch columns (k+1 channels) for the sketch, scoring and
 *   subtraction calls.  The histogram calls (sb_build_histograms,
 *   sb_grow_tree and their sb_workspace_bytes sizes) take k <= 23 (at most
 *   24 channels) and return SB_E_UNSUPPORTED (sizes: -1) above that.  The
 *   paper leaves k free (Section 3); its experiments use k <= 20.
 *
 * Data layouts (device memory; the layouts are this library's choice, made
 * so that each kernel reads whole cache lines of what it needs)
 * ----------------------------------------------------------------------
 * - QUAD-MAJOR BINS (bins4, ld4): the uint32 word q of row i is
 *   bins4[q*ld4 + i], ld4 >= n, and its byte u (little-endian) is the bin of
 *   feature 4q+u.  A row has Q = ceil(m/4) words; bytes of features >= m are
 *   ignored.  The histogram kernel reads this layout: the 64 lanes of a wave
 *   take 64 consecutive rows and read 256 contiguous bytes per word.
 * - COLUMN-MAJOR BINS (bins_cm, ld_cm): the bin of (row i, feature f) is the
 *   byte bins_cm[f*ld_cm + i], ld_cm >= n.  The partition reads it: the rows
 *   of a node are read in one run of the split feature's column.
 * - ROW RECORDS (rec, ld_rec): row i's m bins are the bytes rec[i*ld_rec ..
 *   i*ld_rec + m-1]; ld_rec >= m, ld_rec % 16 == 0, 16-byte aligned base.
 *   The histograms of the deeper levels read it through row indices: one
 *   row is one contiguous record (one 128-byte line for m <= 128 with
 *   ld_rec = 128).
 * - ROW-MAJOR SKETCH (GH, ld_gh): channel t of row i is GH[i*ld_gh + t],
 *   ld_gh >= k+1 floats, 16-byte aligned base.  Channels 0..k-1 are the
 *   sketch columns, channel k is the hessian weight h.  With ld_gh a multiple
 *   of 8 every row fills whole 32-byte sectors, which sb_sketch writes in
 *   full (floats k+1 .. ld_gh-1 are written as 0).
 * sb_layout_bins() builds the three bin layouts from a row-major matrix.
 */
#ifndef SB_H_
#define SB_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SB_ABI_VERSION 4

/* Status codes. */
enum {
  SB_OK = 0,
  SB_E_ARG = 1,          /* bad scalar or missing pointer */
  SB_E_SHAPE = 2,        /* inconsistent sizes, strides or alignment */
  SB_E_UNSUPPORTED = 3,  /* unknown sketch kind or size outside the supported range */
  SB_E_DEVICE = 4        /* a HIP launch or runtime call failed */
};

/* Sketch kinds (Section 3). */
enum {
  SB_SKETCH_TOP_OUTPUTS = 0,       /* Section 3.1 */
  SB_SKETCH_RANDOM_SAMPLING = 1,   /* Section 3.2 */
  SB_SKETCH_RANDOM_PROJECTION = 2, /* Section 3.3 */
  SB_SKETCH_IDENTITY = 3           /* k == d: full-output scoring (no sketch) */
};

/* Call identifiers for sb_workspace_bytes(). */
enum {
  SB_CALL_SKETCH = 0,
  SB_CALL_BUILD_HISTOGRAMS = 1,
  SB_CALL_SCORE_SPLITS = 2,
  SB_CALL_PARTITION_ROWS = 3,
  SB_CALL_GROW_TREE = 4,
  SB_CALL_HIST_EXPONENTS = 5,
  SB_CALL_LEAF_VALUES = 6,
  SB_CALL_GRADIENTS = 7,
  SB_CALL_UPDATE_PREDICTIONS = 8,
  SB_CALL_UPDATE_AND_GRADIENTS = 9
};

/* Losses of sb_gradients (the cross-entropies of the paper's experiments). */
enum {
  SB_LOSS_SOFTMAX_CE = 0,  /* multiclass: softmax cross-entropy, one label per row */
  SB_LOSS_SIGMOID_BCE = 1  /* multilabel: binary cross-entropy per output, sigmoid link */
};

/* Text of the last non-OK status returned on this thread ("" if none). */
const char* sb_last_error(void);

/* SB_ABI_VERSION of the loaded library. */
int32_t sb_abi_version(void);

/*
 * Workspace bytes needed by one call.  Arguments not used by a call are
 * ignored (pass 0).  n: rows (every call that takes rows, BUILD_HISTOGRAMS
 * included).  n_nodes: nodes of the level (BUILD_HISTOGRAMS,
 * SCORE_SPLITS, PARTITION_ROWS), leaves (LEAF_VALUES).  depth: tree depth
 * (GROW_TREE).  d: output dimension (SKETCH, LEAF_VALUES, GRADIENTS,
 * UPDATE_AND_GRADIENTS; the LEAF_VALUES size covers all three hessian
 * forms).  UPDATE_PREDICTIONS needs only n.  Returns -1 (and sets the error
 * text) for sizes outside the range the call itself accepts (n < 2^31, m and
 * d <= 65535, k <= 255, n_bins in [2, 256], nodes as documented per call).
 * sb_layout_bins and sb_subtract_histograms need no workspace.
 */
int64_t sb_workspace_bytes(int32_t call, int64_t n, int32_t m, int32_t n_bins, int32_t d, int32_t k,
                           int32_t n_nodes, int32_t depth);

/*
 * sb_layout_bins -- the three bin layouts from a row-major bin matrix.
 *
 * bins     n x m uint8 bins, row-major: (i, f) at bins[i*ld_bins + f],
 *          ld_bins >= m.  Values must be < n_bins of the later calls.
 * bins4    out (may be NULL): quad-major bins, ld4 >= n.  Bytes of features
 *          >= m are written as 0.
 * bins_cm  out (may be NULL): column-major bins, ld_cm >= n.
 * rec      out (may be NULL): row records, ld_rec % 16 == 0, ld_rec >= m,
 *          16-byte aligned.  Only bytes 0..m-1 of each record are written.
 * Setup work, once per dataset (not on the per-tree path).
 */
int32_t sb_layout_bins(const uint8_t* bins, int64_t n, int32_t m, int64_t ld_bins, uint32_t* bins4, int64_t ld4,
                       uint8_t* bins_cm, int64_t ld_cm, uint8_t* rec, int64_t ld_rec, void* stream);

/*
 * sb_sketch -- build the sketch GH = [G_k, h] (Section 3).
 *
 * G       n x d gradient matrix, column-major: element (i, j) at G[j*ld_g + i],
 *         ld_g >= n.
 * h       n hessian weights (the denominator weights of S; 1 for the
 *         hessian-free score of Section 3).
 * kind    SB_SKETCH_*.
 *   TOP_OUTPUTS      k columns of largest ||g_j||^2 (ties: lower j first),
 *                    scale 1 (Section 3.1).  1 <= k <= d.
 *   RANDOM_SAMPLING  k i.i.d. draws with p_j = ||g_j||^2 / sum_l ||g_l||^2
 *                    (Section 3.2).  Draw t takes the first j with
 *                    C_j > u[t] * C_{d-1}, where C_j is the left-to-right fp64
 *                    prefix sum of the norms, and scales the column by
 *                    fp32(sqrt(C_{d-1} / (k * ||g_j||^2))) = 1/sqrt(k p_j).
 *                    If every column is zero: cols = -1, scales = 0, zero sketch.
 *   RANDOM_PROJECTION G_k = G Pi with Pi the given d x k matrix (Section 3.3;
 *                    the paper draws its entries i.i.d. N(0, 1/k)).  fp32
 *                    accumulation.  cols / scales / norm2 are not written.
 *   IDENTITY         k == d, GH = [G, h].
 * u       RANDOM_SAMPLING only: k uniforms in [0, 1) (fp64, device).  The
 *         paper fixes the distribution of the draws (Section 3.2), not a
 *         generator; the random numbers are an input so that results are
 *         reproducible and can be checked draw by draw.
 * Pi      RANDOM_PROJECTION only: d x k, row-major (Pi[j*k + t]), fp32.
 * GH      out: row-major sketch, ld_gh >= k+1 floats per row, 16-byte aligned:
 *         GH[i*ld_gh + t] = fp32(G[i, cols[t]] * scales[t]) for t < k (one
 *         fp32 multiply; the projection sum for RANDOM_PROJECTION),
 *         GH[i*ld_gh + k] = h[i], and GH[i*ld_gh + t] = 0 for k < t < ld_gh.
 * cols, scales  out (not RANDOM_PROJECTION): k entries each.
 * norm2   out: d fp64 squared column norms; required for TOP_OUTPUTS and
 *         RANDOM_SAMPLING, optional (may be NULL) for IDENTITY, ignored for
 *         RANDOM_PROJECTION.
 * qexp    out: k+1 exponents for the fixed-point histogram accumulation of
 *         sb_build_histograms (same rule as sb_hist_exponents).
 */
int32_t sb_sketch(int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                  const double* u, const float* Pi, float* GH, int64_t ld_gh, int32_t* cols, float* scales,
                  double* norm2, int32_t* qexp, void* ws, int64_t ws_bytes, void* stream);

/*
 * sb_sketch_given_norms -- sb_sketch with the squared column norms of G as an
 * INPUT (norm2: d fp64 values, for example from sb_gradients), so that G is
 * not read for them.  TOP_OUTPUTS and RANDOM_SAMPLING rank and draw by these
 * values; the other kinds ignore them.  Every other argument, output and rule
 * is that of sb_sketch; the workspace size is sb_sketch's.
 */
int32_t sb_sketch_given_norms(int32_t kind, const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h,
                              int32_t k, const double* u, const float* Pi, float* GH, int64_t ld_gh, int32_t* cols,
                              float* scales, const double* norm2, int32_t* qexp, void* ws, int64_t ws_bytes,
                              void* stream);

/*
 * sb_sketch_sparse_projection -- Random Projections (Section 3.3) with a
 * sparse Pi.  The paper notes that the entries of Pi may follow other
 * distributions than the normal one (Achlioptas) and that sparse JL
 * transforms compute G Pi faster (end of the proof of Prop. A.5).
 *
 * Pi (d x k) is passed row-sparse: row j holds s entries, entry q of value
 * pi_val[j*s + q] in column pi_col[j*s + q]; columns outside [0, k) hold
 * nothing (padding), repeated columns add.  s is 1, 2, 4 or 8.
 * GH, ld_gh, h, qexp: as sb_sketch with RANDOM_PROJECTION:
 *   GH[i*ld_gh + t] = sum_j G[i, j] Pi[j, t] in fp32, GH[i*ld_gh + k] = h[i],
 *   padding written as 0.
 * Every column of G is read once.  With s = 1 the product takes 2 n d
 * flops, added in column order; with s = 2, 4 or 8 Pi is first assembled
 * densely in the workspace (entries of a row added in q order in fp32) and
 * multiplied as in sb_sketch, which is faster there.
 * Workspace: sb_workspace_bytes(SB_CALL_SKETCH, ...).
 */
int32_t sb_sketch_sparse_projection(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* h, int32_t k,
                                    int32_t s, const int32_t* pi_col, const float* pi_val, float* GH, int64_t ld_gh,
                                    int32_t* qexp, void* ws, int64_t ws_bytes, void* stream);

/*
 * sb_hist_exponents -- fixed-point exponents for a given GH (row-major).
 *
 * For channel t (t <= k) with M_t = max_i |GH[i*ld_gh + t]|:
 *   qexp[t] = 17 - floor(log2(M_t))   (qexp[t] = 0 if M_t == 0),
 * so every value maps to an integer rint(v * 2^qexp[t]) of magnitude <= 2^18.
 * sb_build_histograms accumulates those integers exactly and reports sums
 * times 2^-qexp[t]; each element therefore contributes an error of at most
 * half a quantum, 2^-(qexp[t]+1) <= 2^-18 M_t.  Exponents must stay fixed
 * for every level of a tree so that sibling subtraction is exact.
 */
int32_t sb_hist_exponents(const float* GH, int64_t n, int64_t ld_gh, int32_t k, int32_t* qexp, void* ws,
                          int64_t ws_bytes, void* stream);

/*
 * sb_build_histograms -- per-node histograms of one tree level (Section 3.4).
 *
 * For every built node j, feature f, channel t <= k and bin b:
 *   H[((j*m + f)*(k+1) + t)*n_bins + b] = sum over the rows r of node j whose
 *       feature f has bin b of channel t of r's sketch,
 * accumulated exactly in fixed point (see sb_hist_exponents) and written as
 * fp64.  The paper does not fix the histogram arithmetic; fixed point makes
 * the sums exact and independent of the order of the adds, so results do
 * not depend on the grid and sibling subtraction is exact.  Nodes not in
 * the build list are left untouched.
 *
 * The bins come from one of two sources, the sketch always from GH
 * (row-major, ld_gh >= k+1, 16-byte aligned, n rows):
 * row_idx == NULL: node j's rows are the positions node_off[j] ..
 *           node_off[j+1]; their bins are read from bins4 (quad-major,
 *           ld4 >= n, 4-byte aligned).  Every load covers contiguous rows.
 *           rec may be NULL.
 * row_idx != NULL: node j's rows are row_idx[node_off[j] .. node_off[j+1]),
 *           each < n; their bins are read from the row records (rec,
 *           ld_rec): one record per row.  bins4 may be NULL.
 * k, qexp   sketch columns and the exponents from sb_sketch.
 * node_off  n_nodes+1 offsets.
 * build_list  n_build node ids to build (NULL = every node; n_build ignored).
 * H         out: [n_nodes][m][k+1][n_bins] fp64.
 * 1 <= k <= 23: more than 24 channels return SB_E_UNSUPPORTED.
 * The call first writes every row's quantised values into its workspace,
 * 16 * ceil((k+1)/6) bytes per row (one 16-byte word per group of six
 * channels), so the workspace grows with n:
 * sb_workspace_bytes(SB_CALL_BUILD_HISTOGRAMS, n, ...).
 */
int32_t sb_build_histograms(const uint32_t* bins4, int64_t ld4, const uint8_t* rec, int64_t ld_rec, int64_t n,
                            int32_t m, int32_t n_bins, const float* GH, int64_t ld_gh, int32_t k,
                            const int32_t* qexp, const int32_t* row_idx, const int32_t* node_off, int32_t n_nodes,
                            const int32_t* build_list, int32_t n_build, double* H, void* ws, int64_t ws_bytes,
                            void* stream);

/*
 * sb_subtract_histograms -- sibling histograms by subtraction.
 *
 * The paper does not use this step: its histogram algorithm (Section 3.4)
 * builds every node.  Since a node's rows are the disjoint union of its two
 * children's rows, every histogram cell of the parent is the sum of the
 * children's cells, so one child follows from the parent and the other.
 * For parent p < n_parents with built child c = build_list[p] (2p or 2p+1):
 *   H_child[c ^ 1] = H_parent[p] - H_child[c]   (all m*n_bins*(k+1) cells).
 * Exact, because histograms are fixed-point sums stored in fp64.  Entries of
 * build_list that are not 2p or 2p+1 leave that pair untouched.
 * H_parent: [n_parents][m][k+1][n_bins]; H_child: [2*n_parents][...], updated
 * in place.
 */
int32_t sb_subtract_histograms(const double* H_parent, double* H_child, int32_t n_parents, int32_t m,
                               int32_t n_bins, int32_t k, const int32_t* build_list, void* stream);

/*
 * sb_score_splits -- best split of every node of a level (Section 2).
 *
 * For node j, feature f and threshold b in [0, n_bins-2], left = bins <= b:
 *   GL_t, HL = prefix sums over bins 0..b; GR_t = T_t - GL_t; HR = T_h - HL;
 *   S = sum_{t<k} GL_t^2/(HL + lambda) + GR_t^2/(HR + lambda),
 * valid iff HL > min_child_weight and HR > min_child_weight.  The best valid
 * candidate maximises S; ties go to the lower f, then the lower b.  Scores
 * are evaluated in fp64.  A node without a valid candidate gets
 * (-1, -1, -inf).  The paper states neither the tie rule nor the treatment
 * of empty children or nodes without a valid split; these are the library's
 * rules.
 * H: [n_nodes][m][k+1][n_bins] fp64.  lambda > 0, min_child_weight >= 0.
 * best_feature, best_bin, best_score: out, n_nodes entries each.
 */
int32_t sb_score_splits(const double* H, int32_t n_nodes, int32_t m, int32_t n_bins, int32_t k, double lambda,
                        double min_child_weight, int32_t* best_feature, int32_t* best_bin, double* best_score,
                        void* ws, int64_t ws_bytes, void* stream);

/*
 * sb_partition_rows -- split every node's rows for the next level.
 *
 * Section 2 (finding the tree structure): the chosen split of leaf R into
 * R_left = {x : x_f <= threshold} and R_right = R minus R_left, applied to
 * every node of the level; the children replace the node as leaves.
 * Node j's rows (row_idx_in[node_off_in[j] .. node_off_in[j+1]), identity
 * order if row_idx_in is NULL) are split stably into left (column-major bin
 * of feature best_feature[j] <= best_bin[j]) then right, written to the same
 * range of row_idx_out.  best_feature[j] < 0 marks a terminal node: every row
 * goes left and the right child is empty.
 * bins_cm, ld_cm  column-major bins (ld_cm >= n).
 * node_off_out    out: 2*n_nodes+1 offsets of the next level.
 * build_list_out  out: n_nodes entries; entry j is the smaller child of node j
 *           (2j on ties), the node whose histogram the next level builds.
 * row_idx_in and row_idx_out must not overlap.
 */
int32_t sb_partition_rows(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm,
                          const int32_t* row_idx_in, const int32_t* node_off_in, int32_t n_nodes,
                          const int32_t* best_feature, const int32_t* best_bin, int32_t* row_idx_out,
                          int32_t* node_off_out, int32_t* build_list_out, void* ws, int64_t ws_bytes,
                          void* stream);

/*
 * sb_partition_rows_noalloc -- sb_partition_rows without a workspace, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).
 *
 * Same arguments, results and checks as sb_partition_rows, minus ws and
 * ws_bytes.  The scratch is a static device array of the library, 8 MiB per
 * device (each GPU the library runs on holds it until the process ends),
 * enough for n up to about 60 million rows: sizes whose workspace
 * (sb_workspace_bytes(SB_CALL_PARTITION_ROWS, ...)) exceeds it return
 * SB_E_UNSUPPORTED before any device work.  The call allocates nothing; its
 * first call on a device looks up that device's copy of the array.  Every
 * call on one GPU shares that array: calls that overlap in time on one GPU
 * (different streams, other host threads) race and must be serialised by the
 * caller.  Nothing in the scratch needs clearing between calls.
 */
int32_t sb_partition_rows_noalloc(const uint8_t* bins_cm, int64_t n, int32_t m, int64_t ld_cm,
                                  const int32_t* row_idx_in, const int32_t* node_off_in, int32_t n_nodes,
                                  const int32_t* best_feature, const int32_t* best_bin, int32_t* row_idx_out,
                                  int32_t* node_off_out, int32_t* build_list_out, void* stream);

/*
 * sb_grow_tree -- the whole level loop for one tree (depth-wise growth).
 *
 * Runs, for level l = 0..depth-1: histograms (all rows at l = 0, bins read
 * from bins4; from l = 1 on, the smaller child of each pair, bins read from
 * the row records), sibling subtraction (fused into the histogram reduction),
 * scoring and partition, entirely on the device with no host
 * synchronisation.
 * bins4 / bins_cm / rec hold the same binned features in the three layouts;
 * GH (row-major) and qexp come from sb_sketch.
 * tree_feature, tree_bin, tree_score: out, 2^depth - 1 entries in level
 *   order (node j of level l at index 2^l - 1 + j).
 * row_idx_out: out, n rows grouped by leaf; leaf_off_out: out, 2^depth + 1
 *   offsets of the leaves (leaf j of the last level owns
 *   row_idx_out[leaf_off_out[j] .. leaf_off_out[j+1])).
 * 1 <= depth <= 12; 1 <= k <= 23 (SB_E_UNSUPPORTED above).
 */
int32_t sb_grow_tree(const uint32_t* bins4, int64_t ld4, const uint8_t* bins_cm, int64_t ld_cm, const uint8_t* rec,
                     int64_t ld_rec, int64_t n, int32_t m, int32_t n_bins, const float* GH, int64_t ld_gh,
                     int32_t k, const int32_t* qexp, int32_t depth, double lambda,
                     double min_child_weight, int32_t* tree_feature, int32_t* tree_bin, double* tree_score,
                     int32_t* row_idx_out, int32_t* leaf_off_out, void* ws, int64_t ws_bytes, void* stream);

/*
 * sb_leaf_values -- leaf values of a grown tree from the full gradient matrix
 * (Section 2, "Finding the leaf values", eq. 3; Section 3: the sketch only
 * serves the structure search, leaf values use all d outputs).
 *
 * For leaf L (rows row_idx[leaf_off[L] .. leaf_off[L+1])) and output j:
 *   V[L*ld_v + j] = -sum_{i in L} G[i, j] / (sum_{i in L} h_ij + lambda),
 * the minimiser of the leaf's second-order objective with diagonal Hessians.
 * G        n x d gradients, column-major: (i, j) at G[j*ld_g + i], ld_g >= n.
 * hess     per-element hessians h_ij, column-major like G (hess[j*ld_hess + i],
 *          ld_hess >= n), or NULL.
 * h        per-row hessians h_i used for every output when hess is NULL, or
 *          NULL: then h_ij = 1 and the denominator is the leaf's row count
 *          plus lambda (the weight of the hessian-free score S_G).
 * row_idx, leaf_off  the leaf segments, as sb_grow_tree writes them: row_idx
 *          a permutation of 0..n-1, leaf_off n_leaves+1 non-decreasing offsets
 *          from 0 to n.  1 <= n_leaves <= 4096.
 * lambda   > 0.  Hessians must be >= 0.
 * V        out: n_leaves x d fp64, row-major with ld_v >= d.  Empty leaves get 0.
 * Accumulation is exact integer arithmetic per block of rows plus fp64 sums
 * in a fixed order: results are deterministic.  Each element contributes an
 * error of at most 2^-41 of the largest magnitude of its column within its
 * block of 2048 rows.
 */
int32_t sb_leaf_values(const float* G, int64_t n, int32_t d, int64_t ld_g, const float* hess, int64_t ld_hess,
                       const float* h, const int32_t* row_idx, const int32_t* leaf_off, int32_t n_leaves,
                       double lambda, double* V, int64_t ld_v, void* ws, int64_t ws_bytes, void* stream);

/*
 * sb_gradients -- first and second derivatives of the loss at the current
 * predictions (Section 2, eq. 2), with the squared column norms of G that the
 * sketch ranks and draws by (Sections 3.1, 3.2) summed in the same pass.
 *
 * F        n x d raw scores, column-major: (i, j) at F[j*ld_f + i], ld_f >= n.
 * loss     SB_LOSS_SOFTMAX_CE: labels[i] in [0, d) (int32, n entries; Y
 *            unused).  p = softmax(F_i); g_ij = p_ij - [j == labels[i]],
 *            h_ij = p_ij (1 - p_ij) (the diagonal of the softmax Hessian).
 *          SB_LOSS_SIGMOID_BCE: Y n x d uint8 0/1 targets, column-major with
 *            ld_y >= n (labels unused).  s = sigmoid(F); g_ij = s_ij - Y_ij,
 *            h_ij = s_ij (1 - s_ij).
 * G        out: n x d fp32 gradients, column-major, ld_g >= n.
 * hess     out (may be NULL): n x d fp32 h_ij, column-major, ld_hess >= n.
 * h_row    out (may be NULL): n fp32 row means of h_ij (one weight per row).
 * norm2    out (may be NULL): d fp64 values sum_i G[i, j]^2 of the stored G,
 *          added in a fixed order (deterministic).
 * fp32 arithmetic with the library's expf; labels outside [0, d) give a row
 * without a target column.  F and G must not overlap.
 */
int32_t sb_gradients(int32_t loss, const float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* labels,
                     const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g, float* hess, int64_t ld_hess,
                     float* h_row, double* norm2, void* ws, int64_t ws_bytes, void* stream);

/*
 * sb_leaf_values_from_loss -- sb_leaf_values with the per-element hessians
 * of a cross-entropy formed from G and the targets instead of being read:
 *   SB_LOSS_SOFTMAX_CE:  p = G[i, j] + [j == labels[i]],
 *   SB_LOSS_SIGMOID_BCE: p = G[i, j] + Y[j*ld_y + i],
 *   h_ij = p (1 - p) in fp32,
 * which is the hessian sb_gradients writes, up to the rounding of g
 * (|error| <= 2^-24 per element).  V and every other argument as in
 * sb_leaf_values; workspace: sb_workspace_bytes(SB_CALL_LEAF_VALUES, ...).
 */
int32_t sb_leaf_values_from_loss(int32_t loss, const float* G, int64_t n, int32_t d, int64_t ld_g,
                                 const int32_t* labels, const uint8_t* Y, int64_t ld_y, const int32_t* row_idx,
                                 const int32_t* leaf_off, int32_t n_leaves, double lambda, double* V, int64_t ld_v,
                                 void* ws, int64_t ws_bytes, void* stream);

/*
 * sb_update_predictions -- the model update a_t = a_{t-1} + lr * f_t
 * (Section 2): for every row i in leaf L of the grown tree and output j,
 *   F[j*ld_f + i] = fp32( (double)F[j*ld_f + i] + lr * V[L*ld_v + j] ),
 * the product and the sum in fp64, rounded once.
 * row_idx, leaf_off, n_leaves: the leaf segments as sb_grow_tree writes them
 * (1 <= n_leaves <= 4096).  V: n_leaves x d fp64 leaf values (sb_leaf_values),
 * ld_v >= d.  F is updated in place.
 */
int32_t sb_update_predictions(float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx,
                              const int32_t* leaf_off, int32_t n_leaves, const double* V, int64_t ld_v, double lr,
                              void* ws, int64_t ws_bytes, void* stream);

/*
 * sb_update_and_gradients -- the update of one tree followed by the
 * derivatives at the new scores, the two consecutive steps of the boosting
 * loop (Section 2: a_t = a_{t-1} + lr * f_t, then eq. 2 at a_t).  The result
 * is bit-identical to sb_update_predictions(F, ..., V, ld_v, lr) followed by
 * sb_gradients(loss, F, ...): F is updated in place, and G, hess, h_row and
 * norm2 are those of the updated F.  Every argument means what it means in
 * those two calls, with the same ranges and errors.
 * For the softmax loss with d <= 104 and at most 256 leaves whose lr * V
 * table (n_leaves x (d | 1) doubles) fits 64 KB, the two run as one pass
 * that reads F once; otherwise as the two calls.
 * Workspace: sb_workspace_bytes(SB_CALL_UPDATE_AND_GRADIENTS, n, d).
 */
int32_t sb_update_and_gradients(int32_t loss, float* F, int64_t n, int32_t d, int64_t ld_f, const int32_t* row_idx,
                                const int32_t* leaf_off, int32_t n_leaves, const double* V, int64_t ld_v, double lr,
                                const int32_t* labels, const uint8_t* Y, int64_t ld_y, float* G, int64_t ld_g,
                                float* hess, int64_t ld_hess, float* h_row, double* norm2, void* ws,
                                int64_t ws_bytes, void* stream);

/*
 * Kernel timing for benchmarks.  Between sb_profile_begin() and
 * sb_profile_end() on one host thread, every launch of the histogram kernel
 * (the LDS-accumulation kernel inside sb_build_histograms and sb_grow_tree)
 * is bracketed by a pair of HIP events recorded on the same stream.
 * sb_profile_end() waits for the last event, returns the summed kernel time
 * in milliseconds and the number of launches, and releases the events.
 * Creating events is host-side work; no device memory is allocated.
 */
int32_t sb_profile_begin(void);
int32_t sb_profile_end(double* hist_kernel_ms, int64_t* hist_launches);

#ifdef __cplusplus
}
#endif

#endif /* SB_H_ */
