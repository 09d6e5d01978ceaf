/*
 * cogdl.h -- C ABI of the MI355X (gfx950) library of GNN message-passing
 * operators described in section 2.2 ("Efficient Sparse Operators") of the
 * CogDL paper (arxiv 2103.00959).
 *
 * Graph and feature conventions, for every call below
 *   - The graph is a sparse matrix A in CSR form: rowptr (int32, n_rows + 1
 *     entries, rowptr[0] = 0, non-decreasing, rowptr[n_rows] = nnz), col
 *     (int32, nnz entries, each in [0, n_cols)) and optional per-edge values
 *     val (fp32, nnz entries; NULL means every value is 1).  Row i is the
 *     aggregating node u of Eq. 1 and col[k] the neighbour v whose feature is
 *     gathered.  Columns may be unsorted inside a row and may repeat; repeated
 *     pairs are separate terms.
 *   - Dense features are row-major: X is n_cols x F (one row per node), Y is
 *     n_rows x F; multi-head features are [node][head][d] (H*D per node).
 *     Per-edge, per-head arrays are edge-major: alpha[k * H + h].
 *   - Feature arrays may be fp32, bf16 or fp16 (cogdl_dtype); edge values,
 *     attention scores and alpha are always fp32; accumulation is always fp32;
 *     narrow outputs are rounded to nearest even.
 *
 * Memory and ownership
 *   - Every array argument is a DEVICE pointer owned by the caller; the
 *     library neither frees nor retains it.  Outputs are fully overwritten,
 *     never accumulated into, and must not overlap any input or each other
 *     (an output may hold intermediate values before the call completes).
 *   - Only cogdl_plan_create allocates device memory and only
 *     cogdl_plan_destroy frees it.  The operator calls never allocate.
 *
 * Errors
 *   - Scalars, NULL pointers, dtype codes, alignment-independent layout rules
 *     and plan/graph consistency are checked on the host before anything is
 *     launched; on error the call returns the code, launches nothing and
 *     leaves every output untouched.
 *   - The library trusts the device contents (rowptr[n_rows] == nnz, columns
 *     in range): it does not read device memory to check them.
 *   - Edge ids are int32: nnz may be at most COGDL_MAX_NNZ (2^31 - 4097, which
 *     leaves room for one batch of indices past the last edge); a larger nnz
 *     gives COGDL_ERR_TOO_LARGE.
 *   - A failed launch returns COGDL_ERR_LAUNCH; a device fault surfaces at the
 *     caller's next synchronization.  No C++ exception crosses this ABI.
 *
 * Concurrency and determinism
 *   - Calls are asynchronous on the given HIP stream (0 = default stream).
 *   - A plan holds a workspace for the partial sums of split rows, so at most
 *     one call that uses a given plan may be in flight at a time; give every
 *     concurrent stream its own plan.
 *   - Results are deterministic: the same inputs give the same bits on every
 *     run (no floating-point atomics; split rows are reduced in a fixed order).
 */
#ifndef COGDL_H
#define COGDL_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    COGDL_OK = 0,
    COGDL_ERR_INVALID = 1,   /* bad scalar, NULL pointer or inconsistent sizes */
    COGDL_ERR_DTYPE = 2,     /* unknown or unsupported dtype code */
    COGDL_ERR_PLAN = 3,      /* plan does not match the graph or the feature width */
    COGDL_ERR_NOMEM = 4,     /* device allocation failed (plan creation only) */
    COGDL_ERR_LAUNCH = 5,    /* a kernel launch or HIP runtime call failed */
    COGDL_ERR_TOO_LARGE = 6  /* a size exceeds what the int32 index format (or a static scratch) holds */
} cogdl_status;

#define COGDL_MAX_NNZ 2147479551LL   /* 2^31 - 4097 */

typedef enum { COGDL_F32 = 0, COGDL_BF16 = 1, COGDL_F16 = 2 } cogdl_dtype;

/* Reduce operation phi of Eq. 1 (section 2.2). */
typedef enum { COGDL_REDUCE_SUM = 0, COGDL_REDUCE_MEAN = 1, COGDL_REDUCE_MAX = 2 } cogdl_reduce;

/* Compute (message) operation psi of Eq. 1: the message of edge k to feature f,
 * with w = val[k] (1 when val is NULL) and x = X[col[k], f]. */
typedef enum {
    COGDL_COMPUTE_MUL = 0,   /* w * x */
    COGDL_COMPUTE_ADD = 1,   /* x + w */
    COGDL_COMPUTE_SUB = 2,   /* x - w */
    COGDL_COMPUTE_COPY = 3   /* x (val ignored) */
} cogdl_compute;

/* Activation applied by the epilogues of the layer entry points (after the
 * bias): identity, max(v, 0), or ELU v > 0 ? v : exp(v) - 1. */
typedef enum { COGDL_ACT_NONE = 0, COGDL_ACT_RELU = 1, COGDL_ACT_ELU = 2 } cogdl_act;

/* Backend choice of the workload balancer (section 2.2, the balancer listing). */
typedef enum {
    COGDL_BALANCE_AUTO = 0,            /* data-aware choice, see cogdl_plan_create */
    COGDL_BALANCE_ROW_SPLIT = 1,       /* one work unit per row, rows in order */
    COGDL_BALANCE_NEIGHBOR_GROUP = 2   /* rows cut into neighbour groups of <= group_size edges */
} cogdl_balance;

#define COGDL_MAX_HEADS 64

typedef struct cogdl_plan cogdl_plan;   /* opaque; owns device work lists and workspace */

typedef struct {
    int32_t n_rows;
    int64_t nnz;
    int32_t group_size;
    int32_t max_feat;
    int32_t max_heads;
    int32_t mode;           /* COGDL_BALANCE_ROW_SPLIT or COGDL_BALANCE_NEIGHBOR_GROUP, as chosen */
    int32_t n_units;        /* work units in execution order */
    int32_t n_long_units;   /* leading units with more than 8 edges; the rest run a narrow path */
    int32_t n_split_rows;   /* rows cut into more than one unit */
    int32_t n_partials;     /* partial-sum slots used by split rows */
    int64_t device_bytes;   /* device memory owned by the plan */
} cogdl_plan_info;

/* Human-readable name of a status code (static storage). */
const char *cogdl_status_string(cogdl_status s);

/* Library version as 10000*major + 100*minor + patch. */
int32_t cogdl_version(void);

/* ------------------------------------------------------------------------
 * Workload balancer -- section 2.2, the "workload balance abstraction"
 * listing: a preprocessing step, run once per graph, that inspects the degree
 * distribution, picks the row-split or the neighbour-group backend and emits
 * the auxiliary arrays the aggregation kernels consume.
 *
 * mode AUTO picks ROW_SPLIT when at least 90% of the rows have a degree d with
 * avg/2 <= d <= 2*avg (avg = nnz / n_rows), NEIGHBOR_GROUP otherwise.  In
 * NEIGHBOR_GROUP mode each row with more than group_size edges is cut into
 * consecutive groups of group_size edges (the last one shorter); every such
 * group is reduced into a partial sum that a second, fixed-order pass adds up.
 * Units are executed longest first.  The result of every operator is the same
 * for both modes up to fp32 summation order.
 *
 * rowptr      device, n_rows + 1 int32 (read on `stream` during the build).
 * max_feat    largest feature width F (or H*D) the plan will serve, >= 1.
 * max_heads   largest head count H the plan will serve in the attention calls
 *             (0 if it serves only cogdl_spmm / cogdl_spmm_t), <= COGDL_MAX_HEADS.
 * group_size  neighbour-group size in edges, >= 1; 0 picks it from the graph size:
 *             the power of two at or below nnz / 16384, clamped to [256, 4096]
 *             (large groups mean fewer partial sums, small ones better balance).
 * The build runs asynchronously on `stream`; *out is valid immediately and
 * every later call on the same stream sees the finished plan.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_plan_create(int32_t n_rows, int64_t nnz, const int32_t *rowptr,
                               int32_t max_feat, int32_t max_heads, cogdl_balance mode,
                               int32_t group_size, hipStream_t stream, cogdl_plan **out);

/* Re-run the balancer of an existing plan on a rowptr with the plan's n_rows
 * and nnz (same mode request and group size).  Allocates nothing.  The build
 * never writes past the plan: if the device rowptr holds more edges than the
 * plan was created for (rowptr[n_rows] > nnz, a broken contract the host
 * cannot see), the plan is left empty (no work unit runs) and the next
 * cogdl_plan_query returns COGDL_ERR_PLAN. */
cogdl_status cogdl_plan_rebuild(cogdl_plan *plan, const int32_t *rowptr, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Column-sliced plan (a scheduling refinement of the neighbour-group backend
 * for the MI355X, not part of the paper): in NEIGHBOR_GROUP mode every row
 * with more than slice_min edges is also cut at the boundaries of 8 equal
 * column ranges [s * w, (s + 1) * w), w = ceil(n_cols / 8) (then into groups
 * of at most group_size edges, each a partial sum as above), and the units
 * are executed as 8 lists: the units of column range s form list s, every
 * other unit goes to list row % 8, and each list runs on one XCD, so the
 * feature rows a list gathers come from one eighth of the table and stay in
 * that XCD's L2.  Any row order of columns is accepted (unsorted rows are
 * still cut into 8 contiguous pieces, only without the locality).  Results
 * are those of the plain plan up to fp32 summation order.
 *
 * col         device, nnz int32: the graph's column indices (for the CSC,
 *             the row indices row_t), read during every build.
 * n_cols      number of columns (>= 1 when nnz > 0).
 * slice_min   rows with more edges than this are sliced; 0 picks
 *             COGDL_DEFAULT_SLICE_MIN.
 * group_size  as for cogdl_plan_create, at most 2^24.
 * The creation counts the sliced units of this graph (one host read-back) to
 * size the plan.  cogdl_plan_rebuild_sliced re-runs the balancer on a graph
 * with the plan's n_rows and nnz; if its sliced units would exceed the sizes
 * taken at creation, that build slices no row.  A sliced plan is rebuilt
 * only with cogdl_plan_rebuild_sliced (cogdl_plan_rebuild returns
 * COGDL_ERR_INVALID for it), and serves every call a plain plan serves.
 * ---------------------------------------------------------------------- */
#define COGDL_DEFAULT_SLICE_MIN 128

cogdl_status cogdl_plan_create_sliced(int32_t n_rows, int64_t nnz, const int32_t *rowptr,
                                      const int32_t *col, int32_t n_cols, int32_t max_feat,
                                      int32_t max_heads, cogdl_balance mode, int32_t group_size,
                                      int32_t slice_min, hipStream_t stream, cogdl_plan **out);

cogdl_status cogdl_plan_rebuild_sliced(cogdl_plan *plan, const int32_t *rowptr, const int32_t *col,
                                       hipStream_t stream);

/* Free the plan (synchronizes the device first).  NULL is accepted. */
cogdl_status cogdl_plan_destroy(cogdl_plan *plan);

/* Read the plan's counters back to the host (synchronizes `stream`).
 * Returns COGDL_ERR_PLAN (with *info filled) when the last build found more
 * work units, partial slots or split rows than the plan's capacities, i.e. a
 * rowptr with more than nnz edges; the plan is then empty until a build on a
 * conforming rowptr. */
cogdl_status cogdl_plan_query(const cogdl_plan *plan, hipStream_t stream, cogdl_plan_info *info);

/* Copy the work units, in execution order, to `units` (device, 4 int32 per
 * unit: row, first edge, end edge, partial slot or -1).  `capacity` is the
 * number of units the buffer holds; at most min(capacity, n_units) are
 * written.  Test and inspection aid. */
cogdl_status cogdl_plan_units(const cogdl_plan *plan, int32_t *units, int64_t capacity,
                              hipStream_t stream);

/* ------------------------------------------------------------------------
 * Generalized SpMM -- section 2.2, Eq. 1 with reduce = sum and compute =
 * multiply, i.e. H' = A H:
 *     Y[i, f] = sum_{k = rowptr[i]}^{rowptr[i+1]-1} val[k] * X[col[k], f]
 * X: n_cols x F of x_dtype; Y: n_rows x F of y_dtype (an empty row gives 0).
 * plan: NULL for the plain row-split mapping, else a plan built on this
 * rowptr (same n_rows and nnz) with max_feat >= F.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_spmm(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                        const int32_t *col, const float *val, int32_t F, const void *X,
                        cogdl_dtype x_dtype, void *Y, cogdl_dtype y_dtype,
                        const cogdl_plan *plan, hipStream_t stream);

/* ------------------------------------------------------------------------
 * GSpMM with a choice of reduce and compute -- section 2.2, Eq. 1 (the user
 * picks the reduce phi and the message psi).  With m_kf the message of edge
 * k (cogdl_compute) and d_i the number of edges of row i:
 *   SUM : Y[i, f] = sum_k m_kf        (MUL: = cogdl_spmm)
 *   MEAN: Y[i, f] = (1 / d_i) * sum_k m_kf
 *   MAX : Y[i, f] = max_k m_kf (messages rounded once to fp32), and
 *         arg[i, f] = the first edge id k, in CSR order, attaining the max
 * An empty row gives 0 (and arg -1).  Messages and sums are computed in
 * fp32.  arg: device int32 n_rows x F, written for MAX only, may be NULL.
 * MAX supports y_dtype equal to x_dtype or fp32 (COGDL_ERR_DTYPE otherwise);
 * an unknown reduce, compute or act code is COGDL_ERR_INVALID.  Epilogue
 * (the aggregation half of a GCN layer): Y[i, f] = act(Y[i, f] + bias[f]),
 * bias fp32 F entries or NULL, applied to every row (an empty row gives
 * act(bias)).  Other arguments and errors as for cogdl_spmm.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_gspmm(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                         const int32_t *col, const float *val, int32_t F, const void *X,
                         cogdl_dtype x_dtype, void *Y, cogdl_dtype y_dtype, cogdl_reduce reduce,
                         cogdl_compute compute, const float *bias, cogdl_act act, int32_t *arg,
                         const cogdl_plan *plan, hipStream_t stream);

/* ------------------------------------------------------------------------
 * CSR -> CSC transpose of the graph structure, the setup of the backward
 * pass of Eq. 1 (the gradient with respect to H is A^T G).
 *   colptr[j]  = number of edges with col < j           (n_cols + 1 int32)
 *   perm[p]    = CSR edge id stored at CSC slot p       (nnz int32, nullable)
 *   row_t[p]   = row of that edge                       (nnz int32)
 *   val_t[p]   = bit copy of val[perm[p]]               (nnz fp32, nullable;
 *                                                        must be NULL if val is)
 * Inside a column the edges appear in increasing CSR edge id (a stable sort),
 * so every output is unique and reproduced bit for bit.
 * workspace: device scratch of at least the size cogdl_csr_to_csc_workspace
 * reports for these sizes (256-byte aligned); its contents are clobbered.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_csr_to_csc_workspace(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                        size_t *bytes);
cogdl_status cogdl_csr_to_csc(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                              const int32_t *col, const float *val, int32_t *colptr,
                              int32_t *row_t, float *val_t, int32_t *perm, void *workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Allocation-free transpose, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): cogdl_csr_to_csc with the same arguments, outputs and errors,
 * minus the workspace.  Its scratch is a static device array of
 * COGDL_NOALLOC_SCRATCH_BYTES (64 MiB) on each GPU, placed when the library's
 * code object is loaded there and held until the process ends; the call
 * itself allocates nothing.  A graph whose workspace
 * (cogdl_csr_to_csc_workspace) exceeds that size -- about 1.6M edges -- is
 * refused with COGDL_ERR_TOO_LARGE before anything is launched.  All calls on
 * one GPU share its array: calls that overlap in time on one GPU (several
 * streams or threads) race and give undefined results; serialize them.
 * Nothing in the scratch needs to be zero, so a call never depends on what the
 * previous one left there.
 * ---------------------------------------------------------------------- */
#define COGDL_NOALLOC_SCRATCH_BYTES (64ull << 20)

cogdl_status cogdl_csr_to_csc_noalloc(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                      const int32_t *rowptr, const int32_t *col, const float *val,
                                      int32_t *colptr, int32_t *row_t, float *val_t, int32_t *perm,
                                      hipStream_t stream);

/* ------------------------------------------------------------------------
 * Transposed SpMM for the backward pass of Eq. 1:
 *     dX[j, f] = sum_{p = colptr[j]}^{colptr[j+1]-1} val_t[p] * G[row_t[p], f]
 * i.e. dX = A^T G, using the CSC arrays from cogdl_csr_to_csc.  n_rows,
 * n_cols and nnz describe A (not A^T): G is n_rows x F, dX is n_cols x F.
 * plan_t: NULL, or a plan built on colptr (n_cols rows, nnz edges).
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_spmm_t(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *colptr,
                          const int32_t *row_t, const float *val_t, int32_t F, const void *G,
                          cogdl_dtype g_dtype, void *dX, cogdl_dtype dx_dtype,
                          const cogdl_plan *plan_t, hipStream_t stream);

/* ------------------------------------------------------------------------
 * SDDMM + LeakyReLU + edge-wise softmax -- section 2.2: the sampled
 * dense-dense product T = A (.) (P Q^T) and the edge-wise softmax
 *     alpha'_uv = exp(alpha_uv) / sum_{w in N(u)} exp(alpha_uw)
 * taken over the edges of each row u, per head.  The attention score is the
 * additive GAT form (the SDDMM with P = [s_dst, 1], Q = [1, s_src] per head):
 *     t = s_dst[i, h] + s_src[col[k], h],   e = t > 0 ? t : negative_slope * t
 *     alpha[k * H + h] = exp(e - m) / sum_{k' in row i} exp(e' - m)
 * where m is the row maximum of e for head h.
 * s_dst: n_rows x H fp32; s_src: n_cols x H fp32; alpha: nnz x H fp32.
 * 1 <= H <= COGDL_MAX_HEADS.  plan: NULL or a plan with max_heads >= H.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_sddmm_edge_softmax(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                      const int32_t *rowptr, const int32_t *col, int32_t H,
                                      const float *s_dst, const float *s_src,
                                      float negative_slope, float *alpha,
                                      const cogdl_plan *plan, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Fused GAT aggregation: the scores, LeakyReLU and edge softmax above followed
 * by the multi-head SpMM of section 2.2 (one weight per edge and head):
 *     Y[i, h, d] = sum_{k in row i} alpha[k, h] * X[col[k], h, d]
 * alpha never has to reach memory.  With alpha_in != NULL the attention steps
 * are skipped and alpha_in (nnz x H fp32, e.g. a permuted alpha for the
 * backward pass) is used as the weights; s_dst / s_src may then be NULL.
 * With alpha_out != NULL the softmax weights are also written (nnz x H fp32).
 * X: n_cols x (H*D) of x_dtype; Y: n_rows x (H*D) of y_dtype.
 * 1 <= H <= COGDL_MAX_HEADS, D >= 1.  plan: NULL or a plan with
 * max_feat >= H*D and max_heads >= H.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_gat_aggregate(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                 const int32_t *rowptr, const int32_t *col, int32_t H, int32_t D,
                                 const float *s_dst, const float *s_src, float negative_slope,
                                 const float *alpha_in, const void *X, cogdl_dtype x_dtype,
                                 void *Y, cogdl_dtype y_dtype, float *alpha_out,
                                 const cogdl_plan *plan, hipStream_t stream);

/* The same with an epilogue (the aggregation half of a GAT layer):
 * Y[i, h, d] = act(aggregate + bias[h * D + d]), bias fp32 H*D entries or
 * NULL, every row included; act outside cogdl_act is COGDL_ERR_INVALID. */
cogdl_status cogdl_gat_aggregate_act(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                     const int32_t *rowptr, const int32_t *col, int32_t H,
                                     int32_t D, const float *s_dst, const float *s_src,
                                     float negative_slope, const float *alpha_in, const void *X,
                                     cogdl_dtype x_dtype, void *Y, cogdl_dtype y_dtype,
                                     float *alpha_out, const float *bias, cogdl_act act,
                                     const cogdl_plan *plan, hipStream_t stream);

/* The fused GAT aggregation of a GAT layer whose source scores are the
 * projection of the aggregated features (section 2.2's multi-head attention;
 * in a GAT layer s_src = Z a_src per head): instead of reading s_src, each
 * edge's source score is formed from the feature row the aggregation gathers
 * anyway,
 *     s_src[j, h] = sum_d X[j, h, d] * a_src[h, d]      (fp32, in the kernel)
 * and the scores, LeakyReLU, edge softmax and multi-head SpMM follow as in
 * cogdl_gat_aggregate_act.  This spares the random score-row read of every
 * edge (a whole cache line for a 4H-byte row).  a_src: fp32 H x D.  The head's
 * D features must be whole 16-byte vectors (D * element size a multiple of
 * 16) with D / (16 / element size) a power of two, and X and Y 16-byte
 * aligned; other shapes give COGDL_ERR_INVALID (use cogdl_head_scores and
 * cogdl_gat_aggregate_act).  Attention weights are not written (a backward
 * pass takes s_src from cogdl_head_scores and alpha from cogdl_gat_aggregate).
 * The scores are rounded in another order than cogdl_head_scores rounds
 * them, so the two paths agree to rounding, not bit for bit.  Other arguments
 * and errors as for cogdl_gat_aggregate_act. */
cogdl_status cogdl_gat_aggregate_proj(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                      const int32_t *rowptr, const int32_t *col, int32_t H,
                                      int32_t D, const float *s_dst, const float *a_src,
                                      float negative_slope, const void *X, cogdl_dtype x_dtype,
                                      void *Y, cogdl_dtype y_dtype, const float *bias,
                                      cogdl_act act, const cogdl_plan *plan, hipStream_t stream);

/* ------------------------------------------------------------------------
 * The attention layer of cogdl_gat_aggregate_act / _proj for training: Y as
 * there, and instead of alpha (nnz x H) the final softmax state of every
 * row, row_stats[i * 2H + h] = m[i,h] (the row's maximum score) and
 * row_stats[i * 2H + H + h] = 1 / z[i,h] (its normalizer), n_rows x 2H fp32,
 * from which cogdl_gat_backward_stats rebuilds every weight with the same
 * bits as alpha_out would hold (section 2.2: the edge softmax's
 * exp(e - m) / z; an empty row gets m = -inf, 1/z = 1).  Exactly one of
 * s_src (scores given, as cogdl_gat_aggregate_act) and a_src (projected, as
 * cogdl_gat_aggregate_proj, same requirements) is non-NULL; row_stats is
 * required.  COGDL_ERR_INVALID otherwise.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_gat_aggregate_stats(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                       const int32_t *rowptr, const int32_t *col, int32_t H,
                                       int32_t D, const float *s_dst, const float *s_src,
                                       const float *a_src, float negative_slope, const void *X,
                                       cogdl_dtype x_dtype, void *Y, cogdl_dtype y_dtype,
                                       float *row_stats, const float *bias, cogdl_act act,
                                       const cogdl_plan *plan, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Dense layer of the GCN and GAT models that the sparse operators of section
 * 2.2 serve (the feature transform of every layer; the paper's end-to-end
 * inference workload is a 2-layer GCN or GAT):
 *     Y[i, c] = act(sum_j X[i, j] * W[c, j] + bias[c])
 * X: n x k, W: m x k (the out x in weights of the layer), both bf16 or both
 * fp16 (dtype; other codes COGDL_ERR_DTYPE); bias: fp32, m entries, or NULL;
 * Y: n x m of y_dtype.  fp32 accumulation on the matrix cores.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_linear(int64_t n, int32_t k, int32_t m, const void *X, const void *W,
                          cogdl_dtype dtype, const float *bias, cogdl_act act, void *Y,
                          cogdl_dtype y_dtype, hipStream_t stream);

/* Per-head attention scores of a GAT layer (section 2.2, the SDDMM inputs):
 *     s_src[i, h] = sum_d Z[i, h, d] * a_src[h, d],  s_dst likewise with a_dst
 * Z: n x H x D of z_dtype; a_src, a_dst: fp32 H x D; s_src, s_dst: fp32 n x H
 * (either may be NULL, with its vector).  fp32 accumulation. */
cogdl_status cogdl_head_scores(int64_t n, int32_t H, int32_t D, const void *Z,
                               cogdl_dtype z_dtype, const float *a_src, const float *a_dst,
                               float *s_src, float *s_dst, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Activation compression (the paper's activation-compression training, 2-4
 * bits in its evaluation): per-group b-bit quantization with stochastic
 * rounding of an n x F activation array A (fp32 / bf16 / fp16).
 * Each row is cut into groups of `group` consecutive features (a multiple of
 * 64, at least 64; the last group of a row may be shorter); bits in [1, 8].
 * For a group with minimum m and maximum M, s = (2^bits - 1) / (M - m) and the
 * step r = (M - m) / (2^bits - 1) (both 0 when M == m); feature x with flat
 * index e = i * F + f gets the code
 *     q = clamp(floor(fma(x - m, s, u)), 0, 2^bits - 1)        (fp32)
 * where u in [0, 1) is word e mod 4 of Philox4x32-10 at counter
 * (e / 4 mod 2^32, e / 2^34, 0, 0) with key (seed mod 2^32, seed / 2^32),
 * its top 24 bits times 2^-24.  Decoding gives fma(q, r, m), an unbiased
 * estimate of x within one step r.
 * Layout: stats[2g], stats[2g+1] = (m, r) for group g = i * groups_per_row + j;
 * codes: group g owns (group / 64) * bits uint64 words, each block of 64
 * consecutive features being `bits` bit planes (plane p has bit p of the code
 * of feature 64 t + l at bit l; features past the end of the row code 0).
 * cogdl_act_codec_size gives the number of code words and stat floats.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_act_codec_size(int64_t n, int32_t F, int32_t bits, int32_t group,
                                  int64_t *code_words, int64_t *stat_floats);
cogdl_status cogdl_act_compress(int64_t n, int32_t F, const void *A, cogdl_dtype a_dtype,
                                int32_t bits, int32_t group, uint64_t seed, uint64_t *codes,
                                float *stats, hipStream_t stream);
cogdl_status cogdl_act_decompress(int64_t n, int32_t F, int32_t bits, int32_t group,
                                  const uint64_t *codes, const float *stats, void *out,
                                  cogdl_dtype out_dtype, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Dot-product SDDMM -- section 2.2, T = A (.) (P Q^T), per head: for every
 * edge k = (i, col[k]) and head h
 *     out[k * H + h] = sum_d P[i, h, d] * Q[col[k], h, d]
 * P: n_rows x H x D of p_dtype; Q: n_cols x H x D of q_dtype; out: nnz x H
 * fp32 (the structure of A only: edge values are not applied).  fp32
 * accumulation.  plan: NULL or a plan on this rowptr (any max_feat).
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_sddmm_dot(int32_t n_rows, int32_t n_cols, int64_t nnz, const int32_t *rowptr,
                             const int32_t *col, int32_t H, int32_t D, const void *P,
                             cogdl_dtype p_dtype, const void *Q, cogdl_dtype q_dtype, float *out,
                             const cogdl_plan *plan, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Backward of the attention layer of cogdl_gat_aggregate (section 2.2: the
 * SDDMM carries the loss gradient to the attention matrix; the rest is the
 * chain rule through the edge softmax, LeakyReLU and the multi-head SpMM).
 * Given dY = dL/dY (n_rows x H x D) and the forward weights alpha (nnz x H,
 * as written by cogdl_gat_aggregate's alpha_out), for edge k = (i, j):
 *   dalpha[k,h] = sum_d dY[i,h,d] * X[j,h,d]
 *   c[i,h]      = sum_{k in row i} alpha[k,h] * dalpha[k,h]
 *   dscore[k,h] = f * alpha[k,h] * (dalpha[k,h] - c[i,h]),  f = 1 when
 *                 s_dst[i,h] + s_src[j,h] > 0, else negative_slope
 *                 (dL/d of the pre-activation score)
 *   ds_dst[i,h] = sum_{k in row i} dscore[k,h]     (n_rows x H)
 *   ds_src[j,h] = sum_{k: col[k] = j} dscore[k,h]  (n_cols x H)
 *   dX[j,h,:]   = sum_{k: col[k] = j} alpha[k,h] * dY[i,h,:]   (n_cols x H x D)
 * colptr, row_t, perm: the CSC of the same graph from cogdl_csr_to_csc.
 * plan: NULL or a plan on rowptr with max_heads >= H; plan_t: NULL or a plan
 * on colptr with max_feat >= H*D and max_heads >= H.  dalpha and dscore are
 * nnz x H fp32 outputs, each of which may be NULL (not written: a layer's
 * backward needs only ds_dst, ds_src and dX, and dscore is also left in
 * edge_work).  edge_work: caller-owned device scratch of nnz x H x 2
 * floats, 8-byte aligned (NULL allowed only when nnz == 0): the first pass
 * leaves there, per edge k (CSR order) and head h, the pair
 * (alpha[k,h], dscore[k,h]) at floats 2(kH + h) and 2(kH + h) + 1, which the
 * second pass reads through perm (one record per edge instead of two rows);
 * it holds those pairs on return.  fp32 accumulation; every output is
 * overwritten.  Both plans' workspaces and edge_work are used: one call per
 * plan pair and workspace in flight.  COGDL_ERR_INVALID for a missing or
 * misaligned edge_work.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_gat_backward(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                const int32_t *rowptr, const int32_t *col, const int32_t *colptr,
                                const int32_t *row_t, const int32_t *perm, int32_t H, int32_t D,
                                const float *s_dst, const float *s_src, float negative_slope,
                                const float *alpha, const void *X, cogdl_dtype x_dtype,
                                const void *dY, cogdl_dtype dy_dtype, void *dX,
                                cogdl_dtype dx_dtype, float *dalpha, float *dscore, float *ds_dst,
                                float *ds_src, float *edge_work, const cogdl_plan *plan,
                                const cogdl_plan *plan_t, hipStream_t stream);

/* ------------------------------------------------------------------------
 * cogdl_gat_backward with the forward weights rebuilt instead of read:
 * row_stats (n_rows x 2H fp32, as written by cogdl_gat_aggregate_stats on
 * the same graph and scores) replaces alpha, and the first pass forms
 * alpha[k,h] = exp(e - m[i,h]) / z[i,h] from the score e it already gathers
 * s_src for, with the forward's own arithmetic: with the scores the forward
 * was given, every output equals cogdl_gat_backward's on that forward's
 * alpha, bit for bit (the records of edge_work included).  With projected
 * scores, s_src here is the caller's projection (cogdl_head_scores), equal
 * to the forward's up to rounding.  The weights rebuilt are softmax outputs
 * (>= 0).  Everything else as cogdl_gat_backward; COGDL_ERR_INVALID for a
 * missing row_stats.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_gat_backward_stats(int32_t n_rows, int32_t n_cols, int64_t nnz,
                                      const int32_t *rowptr, const int32_t *col,
                                      const int32_t *colptr, const int32_t *row_t,
                                      const int32_t *perm, int32_t H, int32_t D,
                                      const float *s_dst, const float *s_src,
                                      float negative_slope, const float *row_stats, const void *X,
                                      cogdl_dtype x_dtype, const void *dY, cogdl_dtype dy_dtype,
                                      void *dX, cogdl_dtype dx_dtype, float *dalpha,
                                      float *dscore, float *ds_dst, float *ds_src,
                                      float *edge_work, const cogdl_plan *plan,
                                      const cogdl_plan *plan_t, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Kernel tracing (instrumentation, not part of the paper's method).  When
 * enabled, every kernel the library launches is bracketed by two HIP events
 * recorded on its launch stream, so the device time of each launch can be
 * read back.  cogdl_trace_enable(capacity) creates `capacity` event pairs
 * (0 disables tracing and frees them); launches beyond the capacity are not
 * recorded.  cogdl_trace_get synchronizes on the i-th stop event and returns
 * the kernel's name (static storage) and its duration in milliseconds.  The
 * tracer is process-wide and not thread-safe.  Each recorded event pair
 * costs the stream a few microseconds, so a timing run that only needs some
 * kernels restricts the trace with cogdl_trace_filter(names): a
 * comma-separated list of launch names (as cogdl_trace_get reports them);
 * only launches named in it are recorded.  NULL or "" records every launch
 * (the default); the list is copied; names longer than 63 characters or a
 * list longer than 1023 characters give COGDL_ERR_INVALID and leave the
 * filter unchanged.
 * ---------------------------------------------------------------------- */
cogdl_status cogdl_trace_enable(int32_t capacity);
cogdl_status cogdl_trace_filter(const char *names);
cogdl_status cogdl_trace_reset(void);
int32_t cogdl_trace_count(void);
cogdl_status cogdl_trace_get(int32_t i, const char **name, float *ms);

#ifdef __cplusplus
}
#endif

#endif /* COGDL_H */
