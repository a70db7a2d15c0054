/*
 * gcn.h -- C ABI of the MI355X (gfx950) GCN training library (libgcn.so).
 *
 * Method: "Morphling: Fast, Fused, and Flexible GNN Training at Scale"
 * (arXiv 2512.01678).  One GCN layer computes Z = A_hat (H W) + b with
 * A_hat = D^-1/2 (A + I) D^-1/2 (Section III-A), followed by ReLU on hidden
 * layers; the input features go through a sparse product when they are sparse
 * enough (Section IV-B, Algorithm 1).
 *
 * Conventions shared by every call:
 *  - Pointers named d_* are device pointers allocated by the caller.  The
 *    library allocates no device memory of its own and never frees caller
 *    memory; scratch space comes from a caller workspace (d_ws, *ws_bytes).
 *  - Workspace protocol: call with d_ws == NULL to have *ws_bytes set to the
 *    bytes needed (nothing is launched); then call again with a buffer of at
 *    least that size.  A smaller *ws_bytes gives GCN_E_CAPACITY.
 *  - Dense matrices are fp32, row-major, with a row pitch ld >= width given in
 *    elements.  Rows whose pitch is a multiple of 4 and whose base is 16-byte
 *    aligned take the vector path; anything else is still correct.  A buffer
 *    of r rows spans r * ld elements (the vector path may read the columns
 *    between width and ld of the last row); those columns are never written.
 *  - Outputs are overwritten, never accumulated into.
 *  - Every call validates its arguments on the host before it enqueues work
 *    on `stream`; an invalid call launches nothing.  Calls documented as
 *    "blocking" synchronise `stream` before they return; the others are
 *    asynchronous and report launch errors as GCN_E_HIP.
 *  - No exception crosses this interface.  gcn_last_error() returns a
 *    thread-local message describing the last failure on the calling thread.
 *  - Results are deterministic on the default path: it uses no floating-point
 *    atomics, so two runs on the same inputs give bitwise-equal outputs.  The one
 *    exception is the sparse backward without a CSC view (gcn_layer_bwd), an
 *    ablation that adds with fp32 atomics.
 */
#ifndef GCN_H_
#define GCN_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t gcn_status;
enum {
  GCN_OK = 0,
  GCN_E_INVALID = -1,     /* NULL where a buffer is required, negative size, ld < width, ... */
  GCN_E_RANGE = -2,       /* an input edge endpoint outside [0, n) */
  GCN_E_OVERFLOW = -3,    /* a count does not fit the index type */
  GCN_E_CAPACITY = -4,    /* workspace or output capacity too small */
  GCN_E_HIP = -5,         /* the HIP runtime reported an error */
  GCN_E_UNSUPPORTED = -6  /* valid request this library does not implement */
};

enum { GCN_DENSE = 0, GCN_SPARSE = 1 };
enum { GCN_ACT_NONE = 0, GCN_ACT_RELU = 1, GCN_ACT_SOFTMAX_CE = 2 };
enum { GCN_ORDER_AUTO = 0, GCN_TRANSFORM_FIRST = 1, GCN_AGGREGATE_FIRST = 2 };
enum { GCN_EPI_NONE = 0, GCN_EPI_RELU = 1, GCN_EPI_MASK = 2 };
enum { GCN_OP_NN = 0, GCN_OP_NT = 1, GCN_OP_TN = 2 };

/* Human-readable name of a status code (static storage). */
const char* gcn_status_string(gcn_status s);
/* Message of the last failing call on this thread ("" if none). */
const char* gcn_last_error(void);
/* Library ABI version (increments on incompatible changes). */
int32_t gcn_version(void);

/*
 * Row-split plan for long rows of a compressed matrix (graph hubs, or columns of
 * X in its CSC view).  A row with more than GCN_SPLIT_MIN entries is "long": it is
 * cut into chunks of GCN_SPLIT_CHUNK entries (the last may be shorter); the
 * product kernels sum each chunk separately and then add a long row's chunk sums
 * in chunk order, so a hub costs many short work items instead of one long one
 * and the result stays deterministic.  The plan is filled by gcn_build_csr (for
 * the graph) and gcn_feature_stats (for the CSC view) when `rows` is non-NULL;
 * a zeroed plan (rows == NULL) means "no splitting".  rows, owner and order hold
 * `cap` entries and first holds cap + 1.  A long row of len > 2 * GCN_SPLIT_CHUNK
 * entries has ceil(len / GCN_SPLIT_CHUNK) < 1.5 len / GCN_SPLIT_CHUNK chunks, so
 * cap >= 3 * entries / (2 * GCN_SPLIT_CHUNK) + 1 always suffices.
 */
enum { GCN_SPLIT_MIN = 4096, GCN_SPLIT_CHUNK = 2048 };
typedef struct gcn_split {
  int32_t n_long;     /* long rows */
  int64_t n_chunk;    /* chunks over all long rows */
  int64_t cap;        /* capacity of the arrays below (entries) */
  int32_t* rows;      /* device, n_long: long row ids, ascending */
  int64_t* first;     /* device, n_long + 1: first chunk of each long row; first[n_long] = n_chunk */
  int32_t* owner;     /* device, n_chunk: index into rows of each chunk */
  int64_t* order;     /* device, n_chunk, or NULL: order in which chunks are processed */
} gcn_split;

/*
 * Graph operator A_hat in CSR form.  Row i lists the distinct neighbours of
 * node i plus i itself, columns ascending; deg[i] is the row length and
 * dinv[i] = (float)(1 / sqrt((double)deg[i])).  val holds the entries of
 * A_hat = D^-1/2 (A + I) D^-1/2 (Section III-A) in CSR order:
 * val[e] = dinv[i] * dinv[col_idx[e]], one fp32 rounding.  The values are
 * computed once, when the graph is built, so an aggregation reads each entry's
 * weight beside its column index instead of gathering dinv of the neighbour.
 */
typedef struct gcn_graph {
  int32_t n;          /* nodes */
  int64_t nnz;        /* entries of A + I (set by gcn_build_csr) */
  int64_t nnz_cap;    /* capacity of col_idx in entries */
  int64_t* row_ptr;   /* device, n + 1 */
  int32_t* col_idx;   /* device, nnz_cap */
  int32_t* deg;       /* device, n */
  float* dinv;        /* device, n */
  float* val;         /* device, nnz_cap: A_hat entries (set by gcn_build_csr) */
  gcn_split split;    /* hub rows (optional; see gcn_split) */
  int32_t* order;     /* device, n, or NULL: the order in which the aggregations over the
                         graph take the rows.  When non-NULL on entry to gcn_build_csr it is
                         written: rows by decreasing length class (4 classes per power of two
                         of the degree), ties in row order, so that the long rows start first
                         and the short ones fill the end of each launch.  Every result is the
                         same, bit for bit, with or without it; NULL takes rows 0 .. n-1. */
} gcn_graph;

/*
 * Input features X (n x f) in compressed form for the sparse path
 * (Algorithm 1: X_csr for Forward, X_csc for Backward).  Values are copied
 * from X bit for bit; rows (CSR) and columns (CSC) list indices ascending.
 */
typedef struct gcn_sparse_x {
  int32_t n, f;
  int64_t nnz;        /* entries; on input to gcn_feature_stats: the capacity */
  int64_t* row_ptr;   /* device, n + 1 */
  int32_t* col;       /* device, nnz */
  float* val;         /* device, nnz */
  int64_t* col_ptr;   /* device, f + 1; NULL: no CSC view */
  int32_t* row;       /* device, nnz */
  float* cval;        /* device, nnz */
  gcn_split csc_split;  /* long columns of the CSC view (optional; see gcn_split) */
} gcn_sparse_x;

/* Density probe result (Section IV-B). */
typedef struct gcn_feature_info {
  int64_t nnz;        /* entries with x != 0.0f (-0.0 is zero, NaN is nonzero) */
  double sparsity;    /* s = 1 - nnz / (n f), for display */
  int32_t mode;       /* GCN_SPARSE iff s >= tau (exact integer test), else GCN_DENSE */
} gcn_feature_info;

/* One GCN layer l: Z = A_hat (H W) + b, H_out = act(Z). */
/*
 * Neighbourhood aggregators (Section III-A: GCN's normalised mean, GIN's sum,
 * mean and max; Listing 1 trains with "Max").  All aggregate over the CSR row of
 * A + I, the node itself included:
 *   GCN_AGG_NORM    A_hat = D^-1/2 (A + I) D^-1/2  (the default)
 *   GCN_AGG_SUM     A + I                           (GIN with epsilon = 0)
 *   GCN_AGG_MEAN    D^-1 (A + I)
 *   GCN_AGG_MEAN_T  (A + I) D^-1, the transpose of the mean (its gradient;
 *                   gcn_aggregate only)
 *   GCN_AGG_MAX     elementwise max over the row, with the first (lowest-column)
 *                   maximiser saved for the gradient
 * A linear aggregator commutes with W, so its layer may run either order; a max
 * layer is always aggregate-first: Z = max-aggregate(H_in) W + b.
 */
enum { GCN_AGG_NORM = 0, GCN_AGG_SUM = 1, GCN_AGG_MEAN = 2, GCN_AGG_MEAN_T = 3, GCN_AGG_MAX = 4 };

typedef struct gcn_layer {
  int32_t f_in, f_out;  /* widths of H_in and H_out */
  int64_t ld_in;        /* pitch of H_in and of the saved aggregate of H_in (aggregate-first) */
  int64_t ld_out;       /* pitch of H_out / Z and of G = dLoss/dZ */
  int32_t act;          /* GCN_ACT_RELU (hidden), GCN_ACT_NONE, GCN_ACT_SOFTMAX_CE (last);
                           gcn_epoch takes ReLU on every hidden layer (GCN_E_UNSUPPORTED
                           otherwise) and softmax cross-entropy on the last */
  int32_t order;        /* GCN_ORDER_AUTO or a forced evaluation order */
  int32_t index;        /* layer number l (0 = input layer) */
  int32_t agg;          /* GCN_AGG_NORM (0), GCN_AGG_SUM, GCN_AGG_MEAN or GCN_AGG_MAX */
} gcn_layer;

/*
 * gcn_build_csr -- A + I from an edge list (Section III-A).  Blocking.
 *
 * d_src, d_dst: n_edges int32 endpoints each (device).  Every pair (u, v) with
 * u != v adds u-v in both directions; pairs with u == v are ignored; repeated
 * pairs count once; each node gets one self-loop.  On entry g->n, g->nnz_cap
 * and the five device pointers must be set; nnz_cap = 2 n_edges + n always
 * suffices.  On return g->nnz holds the entry count.  When g->split.rows is
 * non-NULL the hub split plan is built too (g->split.order is left NULL); when
 * g->order is non-NULL the row order is written (see gcn_graph).
 * Errors: GCN_E_RANGE if an endpoint is outside [0, n) (outputs undefined),
 * GCN_E_CAPACITY if nnz > nnz_cap or the workspace is short.
 */
gcn_status gcn_build_csr(int32_t n, int64_t n_edges, const int32_t* d_src, const int32_t* d_dst,
                         gcn_graph* g, void* d_ws, size_t* ws_bytes, hipStream_t stream);

/*
 * gcn_feature_stats -- density probe, path decision and sparse views
 * (Section IV-B "Sparsity Decision Model" and "Static Path Selection";
 * Algorithm 1, Initialize).  Blocking.
 *
 * Always: counts x != 0.0f per row (into d_row_nnz when non-NULL, int64 n),
 * fills *info: nnz, s = 1 - nnz/(n f), and mode = GCN_SPARSE iff
 * tau_den (n f - nnz) >= tau_num n f, i.e. s >= tau = tau_num / tau_den (the
 * paper's tau is about 0.8: pass 4, 5).  force_mode = GCN_DENSE / GCN_SPARSE
 * overrides the decision; -1 keeps it.
 * When x != NULL it also materialises X_csr (DenseToCSR) and, if x->col_ptr
 * != NULL, X_csc (DenseToCSC); x->nnz must hold the capacity on entry and
 * holds nnz on return.  GCN_E_CAPACITY if the capacity is short.  When
 * x->csc_split.rows is non-NULL, the split plan of the CSC view's long columns is
 * built, with x->csc_split.order (if non-NULL) set to process the chunks
 * chunk-index-major (all columns' first chunks, then all second chunks, ...), so
 * chunks that cover the same window of rows run together.
 */
gcn_status gcn_feature_stats(const float* d_X, int32_t n, int32_t f, int64_t ldx,
                             int32_t tau_num, int32_t tau_den, int32_t force_mode,
                             int64_t* d_row_nnz, gcn_feature_info* info, gcn_sparse_x* x,
                             void* d_ws, size_t* ws_bytes, hipStream_t stream);

/* Evaluation order the library uses for a layer: GCN_TRANSFORM_FIRST
 * (S (H W)) or GCN_AGGREGATE_FIRST ((S H) W) for the layer's aggregator S.  For
 * a linear aggregator both are the same product and the cheaper one aggregates
 * fewer columns per epoch; a max layer is always aggregate-first.  x_sparse: the
 * layer's input is sparse X. */
int32_t gcn_layer_order(const gcn_layer* L, int32_t x_sparse);

/*
 * gcn_layer_fwd -- forward pass of one layer (Section III-A update;
 * Algorithm 1, Forward).  Asynchronous.
 *
 * Exactly one of d_Hin (dense n x f_in, pitch ld_in) and x (sparse input
 * features, layer 0 only) is non-NULL.  d_W: f_in x f_out, pitch f_out.
 * d_b: f_out.  Output d_Hout (n x f_out, pitch ld_out):
 *   GCN_ACT_RELU: H_out = max(Z, 0);  GCN_ACT_NONE: Z;
 *   GCN_ACT_SOFTMAX_CE: G = (softmax(Z) - onehot(labels)) / n, and *d_loss
 *   (device fp32 scalar) = (1/n) sum_i (logsumexp(Z_i) - Z_i,labels_i);
 *   d_labels: n int32 in [0, f_out).  The logits themselves are written to
 *   d_logits (pitch ld_out) when it is non-NULL.
 * The aggregator is L->agg (A_hat for GCN_AGG_NORM).
 * d_saved: n x f_in (pitch ld_in), receives the aggregate S H_in when the layer
 * is evaluated aggregate-first (needed again by gcn_layer_bwd); may be NULL
 * otherwise.  A max layer needs twice that: the maxima (n x ld_in fp32), then the
 * maximisers (n x ld_in int32 node ids) at d_saved + n * ld_in.  A max layer takes
 * dense input only (GCN_E_UNSUPPORTED for sparse X) and f_in <= 256.
 */
gcn_status gcn_layer_fwd(const gcn_graph* g, const gcn_layer* L, const float* d_Hin,
                         const gcn_sparse_x* x, const float* d_W, const float* d_b,
                         float* d_Hout, float* d_saved, const int32_t* d_labels, float* d_loss,
                         float* d_logits, void* d_ws, size_t* ws_bytes, hipStream_t stream);

/*
 * gcn_layer_bwd -- backward pass of one layer (Algorithm 1, Backward).
 * Asynchronous.
 *
 * d_G = dLoss/dZ (n x f_out, pitch ld_out).  Writes d_dW = dLoss/dW (f_in x
 * f_out, pitch f_out) and d_db = sum_i G[i,:] (f_out).  With Q = S^T G (A_hat
 * and A + I are symmetric; the mean's transpose is (A + I) D^-1): dW = H_in^T Q,
 * or X^T Q on the sparse path: gathered through X_csc when x has the CSC view, else
 * (x->col_ptr == NULL, which saves the CSC memory) by atomic adds from the rows of
 * X_csr, the implicit transpose of Section IV-D, whose rounding order is not fixed
 * (results vary within fp32 rounding from run to run; f_out <= 256).  When d_Gprev != NULL (layers above the
 * first) it receives the gradient of the previous layer's pre-activation:
 * (Q W^T) * 1[H_in > 0] (n x f_in, pitch ld_in).  Max layers: dW = P^T G with the
 * saved maxima P, and G_prev routes (G W^T)[u,c] to the saved maximiser of (u, c).
 * d_saved is the buffer gcn_layer_fwd filled for aggregate-first layers.
 */
gcn_status gcn_layer_bwd(const gcn_graph* g, const gcn_layer* L, const float* d_G,
                         const float* d_Hin, const gcn_sparse_x* x, const float* d_saved,
                         const float* d_W, float* d_dW, float* d_db, float* d_Gprev,
                         void* d_ws, size_t* ws_bytes, hipStream_t stream);

/*
 * Whole model for gcn_epoch.  Host arrays of n_layers device pointers each.
 * act[l] (l < n_layers - 1) holds H_{l+1}; grad[l] holds G_l = dLoss/dZ_l;
 * saved[l] holds the aggregate of H_l for aggregate-first layers (twice that
 * size for max layers, see gcn_layer_fwd; NULL entries allowed otherwise).  Adam state m*, v* starts at zero; step counts completed steps.
 */
typedef struct gcn_model {
  int32_t n_layers;
  const gcn_layer* layers;
  float** W;
  float** b;
  float** dW;
  float** db;
  float** mW;
  float** vW;
  float** mb;
  float** vb;
  float** act;
  float** saved;
  float** grad;
  double lr, beta1, beta2, eps;  /* Adam hyperparameters (the paper: 0.01, 0.9, 0.999) */
  int32_t step;
  int32_t* d_step;  /* optional device counter of completed steps; see gcn_epoch */
} gcn_model;

/*
 * gcn_epoch -- one full-batch training epoch (Listing 1): forward through all
 * layers, softmax cross-entropy over all n nodes, backward in reverse, then
 * one Adam step (bias-corrected, step t = m->step + 1) over every W and b.
 * Asynchronous; increments m->step on success.  Exactly one of d_X (dense,
 * pitch m->layers[0].ld_in) and x (sparse path) is non-NULL.  *d_loss receives
 * the mean loss of the forward pass.  When m->d_step is non-NULL the step number
 * is read from and incremented in device memory instead (m->step is left alone),
 * so the enqueued work depends on no host value that changes between epochs and
 * one epoch can be captured in a HIP graph and replayed.  No call made by an
 * epoch allocates, synchronises or records a memset.
 */
gcn_status gcn_epoch(gcn_model* m, const gcn_graph* g, const float* d_X, const gcn_sparse_x* x,
                     const int32_t* d_labels, float* d_loss, void* d_ws, size_t* ws_bytes,
                     hipStream_t stream);

/* ------------------------------------------------------------------------
 * Lower-level steps, exported for unit parity tests and per-kernel timing.
 * ---------------------------------------------------------------------- */

/*
 * gcn_aggregate -- Z = S M (+ b) over all n rows, S = A_hat (GCN_AGG_NORM), A + I
 * (GCN_AGG_SUM), D^-1 (A + I) (GCN_AGG_MEAN) or (A + I) D^-1 (GCN_AGG_MEAN_T)
 * (Section III-A; Algorithm 3's row-parallel, atomic-free aggregation).  Asynchronous.
 * d_M: n x w (pitch ldm).  d_bias: w or NULL.  epi: GCN_EPI_NONE, GCN_EPI_RELU
 * (max(Z, 0)) or GCN_EPI_MASK (Z * 1[mask > 0], d_mask n x w, pitch ldmask).
 * d_Z: n x w (pitch ldz); must not overlap d_M.  The workspace holds the chunk
 * sums of split hub rows (g->split.n_chunk x w floats, rounded up).
 */
gcn_status gcn_aggregate(const gcn_graph* g, int32_t agg, int32_t w, const float* d_M, int64_t ldm,
                         const float* d_bias, int32_t epi, const float* d_mask, int64_t ldmask,
                         float* d_Z, int64_t ldz, void* d_ws, size_t* ws_bytes, hipStream_t stream);

/*
 * gcn_aggregate_max -- max aggregation (GCN_AGG_MAX): P[u,c] = max over the row
 * of A + I of M[v,c] and arg[u,c] = the first v (lowest column) attaining it.
 * Asynchronous.  d_M: n x w (pitch ldm); d_P: n x w fp32 (pitch ldp); d_arg:
 * n x w int32 (pitch ldarg).  w <= 256 (64 when a pitch is not a multiple of 4 or
 * a buffer is not 16-byte aligned): else GCN_E_UNSUPPORTED.  No workspace (the
 * size query returns 0).
 */
gcn_status gcn_aggregate_max(const gcn_graph* g, int32_t w, const float* d_M, int64_t ldm, float* d_P,
                             int64_t ldp, int32_t* d_arg, int64_t ldarg, void* d_ws, size_t* ws_bytes,
                             hipStream_t stream);

/*
 * gcn_aggregate_max_bwd -- gradient of the max aggregation: dM[u,c] = sum over
 * v in the row of u of dP[v,c] * [arg[v,c] == u] (A + I is symmetric, so this
 * gathers every output that u supplied), times 1[mask[u,c] > 0] when d_mask is
 * non-NULL.  Asynchronous; fixed summation order, no atomics.  d_dP, d_arg as
 * produced with gcn_aggregate_max (n x w); d_dM: n x w (pitch ldo), must not
 * overlap the inputs.  Same width limits; no workspace.
 */
gcn_status gcn_aggregate_max_bwd(const gcn_graph* g, int32_t w, const float* d_dP, int64_t ldd,
                                 const int32_t* d_arg, int64_t ldarg, const float* d_mask, int64_t ldmask,
                                 float* d_dM, int64_t ldo, void* d_ws, size_t* ws_bytes, hipStream_t stream);

/*
 * gcn_gemm -- dense fp32 product on the matrix cores (the dense-path GEMM of
 * Algorithm 1).  Asynchronous.
 *   GCN_OP_NN: C (m x n) = A (m x k, pitch lda) B (k x n, pitch ldb)
 *   GCN_OP_NT: C (m x n) = A (m x k) B^T, B is n x k (pitch ldb)
 *   GCN_OP_TN: C (m x n) = A^T B, A is k x m (pitch lda), B is k x n
 * Epilogue: d_bias (n, or NULL) is added, then epi applies (GCN_EPI_RELU, or
 * GCN_EPI_MASK with d_mask m x n, pitch ldmask).  GCN_OP_TN may split k across
 * workgroups; its partial products live in the workspace and are summed in a
 * fixed order.  GCN_OP_NN / GCN_OP_NT without the mask epilogue, n <= 256 and
 * m >= 32768 (A 16-byte aligned, lda % 4 == 0; GCN_GEMM_ROWS=1 from m >= 128 on,
 * =0 never) split B once into the workspace (3 bf16 planes, about 6 k n bytes)
 * and stream the rows of A; the workspace is then required.
 */
gcn_status gcn_gemm(int32_t op, int64_t m, int64_t n, int64_t k, const float* d_A, int64_t lda,
                    const float* d_B, int64_t ldb, float* d_C, int64_t ldc, const float* d_bias,
                    int32_t epi, const float* d_mask, int64_t ldmask, void* d_ws,
                    size_t* ws_bytes, hipStream_t stream);

/*
 * gcn_gemm_static -- gcn_gemm for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * arguments, kernels and results as gcn_gemm, with the product's scratch (split-k partial
 * tiles, the split weight planes of the row-panel product) taken from a static device
 * array of GCN_STATIC_WS_BYTES that the library holds on each device it runs on, instead
 * of from a caller workspace.  Allocates nothing.  GCN_E_CAPACITY (nothing launched) when
 * the product needs more scratch than that; gcn_gemm's size query gives the need.  All
 * calls on one device share its array: calls that overlap on one device (several streams
 * or threads) race and must be serialised by the caller.  Asynchronous.
 */
#define GCN_STATIC_WS_BYTES (64ll << 20)
gcn_status gcn_gemm_static(int32_t op, int64_t m, int64_t n, int64_t k, const float* d_A, int64_t lda,
                           const float* d_B, int64_t ldb, float* d_C, int64_t ldc, const float* d_bias,
                           int32_t epi, const float* d_mask, int64_t ldmask, hipStream_t stream);

/*
 * gcn_spmm -- C[i,:] = sum_e val[e] B[idx[e],:] over compressed rows
 * i < nrows (Section IV-B backend-specialised primitives: X_csr W forward,
 * X^T G from X_csc backward).  Asynchronous.  d_ptr: nrows + 1 int64;
 * nnz: d_ptr[nrows] as known to the host, used only to shape the launch (-1 if
 * unknown); d_idx, d_val: d_ptr[nrows] entries with 0 <= idx < b_rows; d_B: b_rows x w
 * (pitch ldb); d_C: nrows x w (pitch ldc).  split: plan of the long rows of this
 * matrix (or NULL); the workspace holds their chunk sums.
 */
gcn_status gcn_spmm(int64_t nrows, int64_t nnz, const int64_t* d_ptr, const int32_t* d_idx,
                    const float* d_val, int64_t b_rows, int32_t w, const float* d_B, int64_t ldb,
                    float* d_C, int64_t ldc, const gcn_split* split, void* d_ws, size_t* ws_bytes,
                    hipStream_t stream);

/*
 * gcn_spmm_xt -- C = X^T B with X (n x f) in its CSC view: the backward SpMM over
 * X_csc of Algorithm 1 (dW_0 = X^T Q of a sparse first layer).  Asynchronous.
 * d_col_ptr: f + 1 int64; d_row, d_cval: nnz row indices (ascending within a column,
 * 0 <= row < n) and values, as gcn_feature_stats writes them; d_B: n x w (pitch ldb);
 * d_C: f x w (pitch ldc), overwritten.  csc_split: plan of the long columns (or NULL).
 * When the columns hold at least 16 entries per 8,192-row chunk on average and n spans
 * four chunks or more, the rows are cut into such chunks: every (column, chunk) range
 * is summed into a partial in the workspace (the chunk's rows of B stay in one L2) and
 * the partials are added in chunk order; otherwise each column is one gathered sum.
 * GCN_XT=plain / =tiled forces either form.  Deterministic; w <= 256 for the chunked
 * form.  Workspace: query with d_ws == NULL.
 */
gcn_status gcn_spmm_xt(int32_t n, int32_t f, int64_t nnz, const int64_t* d_col_ptr, const int32_t* d_row,
                       const float* d_cval, const gcn_split* csc_split, const float* d_B, int64_t ldb,
                       int32_t w, float* d_C, int64_t ldc, void* d_ws, size_t* ws_bytes, hipStream_t stream);

/*
 * gcn_spmm_xw -- C = X W with X (n x f) in its CSR view: the forward SpMM of a sparse
 * first layer (Algorithm 1, Forward; the product gcn_layer_fwd takes).  Asynchronous.
 * d_row_ptr: n + 1 int64; d_col, d_val: nnz column indices (ascending within a row,
 * 0 <= col < f) and values, as gcn_feature_stats writes them; d_W: f x w (pitch ldw);
 * d_C: n x w (pitch ldc), overwritten.  Lane slices of each row gather a row of W per
 * entry, as the aggregation does (W of the layer stays in L2).  Deterministic.  Needs no
 * workspace (the size query returns 0).
 */
gcn_status gcn_spmm_xw(int32_t n, int32_t f, int64_t nnz, const int64_t* d_row_ptr, const int32_t* d_col,
                       const float* d_val, const float* d_W, int64_t ldw, int32_t w, float* d_C, int64_t ldc,
                       void* d_ws, size_t* ws_bytes, hipStream_t stream);

/*
 * gcn_column_sums -- out[c] = sum_i G[i,c] (the bias gradient) and, when
 * d_row_vals != NULL, *d_mean = (1/rows) sum_i row_vals[i].  Fixed summation
 * order.  Asynchronous.
 */
gcn_status gcn_column_sums(int64_t rows, int32_t w, const float* d_G, int64_t ldg, float* d_out,
                           const float* d_row_vals, float* d_mean, void* d_ws, size_t* ws_bytes,
                           hipStream_t stream);

/* One parameter tensor for gcn_adam. */
typedef struct gcn_adam_tensor {
  float* param;
  const float* grad;
  float* m;
  float* v;
  int64_t count;
} gcn_adam_tensor;

/*
 * gcn_adam -- one bias-corrected Adam step t >= 1 over up to 16 tensors in a
 * single launch (Listing 1 optimizer("adam", lr, beta1, beta2)); the
 * hyperparameters and 1 - beta are formed in double, then rounded to fp32:
 *   m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2;
 *   p -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
 * Asynchronous.
 */
gcn_status gcn_adam(const gcn_adam_tensor* t, int32_t count, int32_t step, double lr, double beta1,
                    double beta2, double eps, hipStream_t stream);

/* As gcn_adam, with the step read from *d_step (completed steps; this step is
 * *d_step + 1) and *d_step incremented on the device afterwards. */
gcn_status gcn_adam_device_step(const gcn_adam_tensor* t, int32_t count, int32_t* d_step, double lr,
                                double beta1, double beta2, double eps, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Kernel timing with HIP events (used by the benchmark).
 * ---------------------------------------------------------------------- */

typedef struct gcn_profile_record {
  char name[64];      /* kernel family, e.g. "aggregate_w256" */
  int32_t width;      /* columns processed */
  int64_t rows;       /* output rows */
  int64_t nnz;        /* sparse entries traversed */
  float ms;           /* elapsed between the events bracketing the launch */
} gcn_profile_record;

/* capacity > 0: start recording events around every aggregation and GEMM
 * launch, up to capacity launches (older records are dropped); 0: stop and
 * release the events.  Host-side only; records events on the launch stream. */
gcn_status gcn_profile_enable(int32_t capacity);
/* Number of records held. */
int32_t gcn_profile_count(void);
/* Record i (0 = oldest); waits for its end event.  GCN_E_INVALID if out of range. */
gcn_status gcn_profile_read(int32_t i, gcn_profile_record* rec);
/* Drop all records (keeps recording enabled). */
gcn_status gcn_profile_reset(void);
/* Record only launches whose family name is exactly `name` (NULL or "": every
 * launch).  Each event pair costs a few microseconds of queue time between
 * kernels, so a timed run brackets only the launches it reports.  The name is
 * copied; at most 63 characters (GCN_E_INVALID beyond). */
gcn_status gcn_profile_only(const char* name);

#ifdef __cplusplus
}
#endif

#endif /* GCN_H_ */
