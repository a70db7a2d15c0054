// internal.h -- declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstdio>
#include <cstdint>
#include <string>

#include "gcn.h"

namespace gcn {

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------
gcn_status fail(gcn_status s, const std::string& msg);
gcn_status hip_fail(hipError_t e, const char* what);
inline gcn_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? GCN_OK : hip_fail(e, what);
}

#define GCN_TRY(expr)                      \
  do {                                     \
    gcn_status _s = (expr);                \
    if (_s != GCN_OK) return _s;           \
  } while (0)

#define GCN_HIP(expr, what)                          \
  do {                                               \
    hipError_t _e = (expr);                          \
    if (_e != hipSuccess) return hip_fail(_e, what); \
  } while (0)

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Sub-allocator over a caller workspace: first pass measures, second pass carves.
struct Arena {
  char* base = nullptr;  // NULL while measuring
  size_t used = 0;
  template <class T>
  T* take(int64_t count) {
    used = (size_t)round_up((int64_t)used, 256);
    T* p = base ? reinterpret_cast<T*>(base + used) : nullptr;
    used += sizeof(T) * (size_t)(count > 0 ? count : 0);
    return p;
  }
};

// ---------------------------------------------------------------------------
// profiling hooks (events around launches; no-ops when disabled)
// ---------------------------------------------------------------------------
struct ProfScope {
  int slot = -1;
  hipStream_t stream = nullptr;
  ProfScope(const char* name, int32_t width, int64_t rows, int64_t nnz, hipStream_t s);
  ~ProfScope();
};

// ---------------------------------------------------------------------------
// launchers (each validates nothing: callers in api.hip validate first)
// ---------------------------------------------------------------------------
enum AggEpi { AGG_NONE = 0, AGG_RELU = 1, AGG_MASK = 2, AGG_SOFTMAX = 3 };
// Entry weights of a linear aggregation over the rows of a compressed matrix:
//   AGG_W_VAL      val[e] (A_hat, or the values of X)
//   AGG_W_ONE      1                      (sum over the row: A + I)
//   AGG_W_ROWMEAN  1, the row sum times 1 / deg[u]  (mean: D^-1 (A + I))
//   AGG_W_COLMEAN  1 / deg[col[e]]        (transpose of the mean: (A + I) D^-1)
enum AggWeight { AGG_W_VAL = 0, AGG_W_ONE = 1, AGG_W_ROWMEAN = 2, AGG_W_COLMEAN = 3 };

struct AggParams {
  int32_t n;               // output rows
  const int64_t* row_ptr;  // n + 1
  const int32_t* col;      // neighbours / column indices
  const float* val;        // entry values (A_hat, or X in CSR / CSC form); kind AGG_W_VAL
  int32_t kind;            // AggWeight: where an entry's weight comes from
  const int32_t* deg;      // row lengths, for the mean kinds
  const float* M;          // gathered rows
  int64_t ldm;
  int32_t w;
  const float* bias;       // w or NULL
  int32_t epi;             // AggEpi
  const float* mask;       // AGG_MASK
  int64_t ldmask;
  float* Z;
  int64_t ldz;
  // softmax cross-entropy epilogue
  const int32_t* labels;
  float* row_loss;         // n: per-row loss
  float* logits;           // optional copy of Z
  int64_t ldl;
  float inv_n;             // 1 / n
  const char* tag;         // kernel family name for the profiler (NULL: derived)
  // AGG_RELU: optional bitmask of the output, bit c % 32 of word c / 32 of a row = 1[Z > 0]
  uint32_t* relu_bits;
  int64_t ld_relu_bits;    // words per row (>= ceil(w / 32))
  // order in which the main kernel takes the rows (n entries), or NULL for 0 .. n-1
  const int32_t* order;
};
// Words per row of a ReLU bitmask of width w.
inline int64_t relu_bits_words(int32_t w) { return (w + 31) / 32; }
// Z over all rows; rows longer than GCN_SPLIT_MIN go through the split plan when one
// is given (its chunk sums live in ws, aggregate_workspace() bytes).
size_t aggregate_workspace(const gcn_split* split, int32_t w);
gcn_status launch_aggregate(const AggParams& p, int64_t nnz, const gcn_split* split, void* ws,
                            hipStream_t s);
inline bool has_split(const gcn_split* sp) { return sp && sp->rows && sp->n_long > 0; }
// Neighbour slices per row for slices of `lanes` lanes on a matrix with nnz entries over
// `rows` rows (nnz < 0: unknown).
int agg_slots(int lanes, int64_t nnz, int64_t rows);
// Max aggregation over the graph rows (P, arg) and its gradient (aggmax.hip).
gcn_status launch_aggregate_max(const AggParams& p, int64_t nnz, float* P, int64_t ldp, int32_t* arg,
                                int64_t ldarg, hipStream_t s);
gcn_status launch_aggregate_max_bwd(const AggParams& p, int64_t nnz, const int32_t* arg, int64_t ldarg,
                                    const float* mask, int64_t ldmask, float* dM, int64_t ldo, hipStream_t s);
// C (out_rows x w) = X^T B from X's CSR rows with atomic adds (C is zeroed first);
// non-deterministic rounding order.  w <= 256.
gcn_status launch_spmm_t_atomic(int64_t nrows, const int64_t* ptr, const int32_t* idx, const float* val,
                                const float* B, int64_t ldb, int32_t w, int64_t out_rows, float* C, int64_t ldc,
                                int64_t nnz, hipStream_t s);
// C (F x w) = X^T B from X's CSC view (col_ptr over F columns, ascending row indices
// in row / values in cval), in row chunks of xt_chunk_rows() rows: each (column, chunk)
// sum goes to a partial, and the partials are added in chunk order.  Deterministic.
// w <= 256.
int64_t xt_chunk_rows();
bool xt_tiled_enabled(int64_t n, int32_t F, int64_t nnz, int32_t w);
size_t xt_tiled_workspace(int64_t n, int32_t F, int32_t w);
gcn_status launch_spmm_xt_tiled(int64_t n, int32_t F, const int64_t* col_ptr, const int32_t* row, const float* cval,
                                int64_t nnz, const float* B, int64_t ldb, int32_t w, float* C, int64_t ldc, void* ws,
                                hipStream_t s);
// X^T B from the CSC view in the form xt_tiled_enabled picks (gcn_spmm_xt).
size_t spmm_xt_workspace(int64_t n, int32_t F, int64_t nnz, int32_t w, const gcn_split* csc_split);
gcn_status launch_spmm_xt(int64_t n, int32_t F, int64_t nnz, const int64_t* col_ptr, const int32_t* row,
                          const float* cval, const gcn_split* csc_split, const float* B, int64_t ldb, int32_t w,
                          float* C, int64_t ldc, void* ws, hipStream_t s);
// C (m x n, pitch ldc) = sum over z < splits of part[z] (m x n, dense), in order of z.
gcn_status launch_partial_sum(const float* part, int64_t splits, int64_t m, int64_t n, float* C, int64_t ldc,
                              hipStream_t s);
// Identity operator in CSR form: row_ptr[i] = i, col[i] = i.
gcn_status launch_identity_csr(int32_t n, int64_t* row_ptr, int32_t* col, hipStream_t s);
// Only the long rows of a split plan (chunk sums, then their combination), no epilogue.
gcn_status launch_aggregate_long_rows(const AggParams& p, const gcn_split* split, void* ws, hipStream_t s);

// Aggregate-first layer in one kernel: P = A_hat X (written to a.Z), H = act(P W + b),
// in the bf16x6 arithmetic of the dense products.  W is f_in x f_out (pitch ldw).
bool agg_gemm_supported(int32_t f_in, int64_t ldx, int64_t ldp, const float* X, const float* P);
size_t agg_gemm_workspace(const gcn_split* split, int32_t f_in, int32_t f_out);
gcn_status launch_agg_gemm(const AggParams& a, int64_t nnz, const gcn_split* split, const float* W,
                           int64_t ldw, int32_t f_out, const float* bias, bool relu, float* H, int64_t ldh,
                           void* ws, hipStream_t s);

// split plan of the long rows of a compressed matrix with offsets ptr[0..nrows]
size_t split_workspace(int64_t nrows);
gcn_status build_split(const int64_t* ptr, int64_t nrows, gcn_split* sp, bool chunk_major, void* ws,
                       hipStream_t s);

enum GemmEpi { GEMM_NONE = 0, GEMM_RELU = 1, GEMM_MASK = 2 };
// C(m,n) = sum_k A(m,k) B(k,n) with A(m,k) = A[m*lda+k] (ta=false) or A[k*lda+m] (ta=true),
// B(k,n) = B[k*ldb+n] (tb=false) or B[n*ldb+k] (tb=true).
struct GemmParams {
  int64_t m, n, k;
  const float* A;
  int64_t lda;
  bool ta;
  const float* B;
  int64_t ldb;
  bool tb;
  float* C;
  int64_t ldc;
  const float* bias;
  int32_t epi;
  const float* mask;
  int64_t ldmask;
  // Bitmask forms (row-panel product only): GEMM_MASK reads bit c % 32 of word c / 32 of
  // row r of mask_bits instead of mask > 0; GEMM_RELU also writes 1[C > 0] to relu_bits.
  const uint32_t* mask_bits = nullptr;
  int64_t ld_mask_bits = 0;
  uint32_t* relu_bits = nullptr;
  int64_t ld_relu_bits = 0;
  // Row-panel product with GEMM_MASK only: also write the column sums of C (n floats,
  // fixed order) -- the bias gradient of the layer below, whose gradient C is.
  float* colsum = nullptr;
  // Row-panel product: B already split into its bf16 planes (launch_split_batch); the
  // product then skips its own split.
  const void* bsplit = nullptr;
};
// Workspace of launch_gemm: split-k partials (A^T B), or the split B of the row-panel
// product (A B, A B^T with n <= 256); 0 when neither applies.
size_t gemm_workspace(const GemmParams& p);
bool gemm_split_k(const GemmParams& p);
bool gemm_rows_supported(const GemmParams& p);
size_t gemm_rows_workspace(const GemmParams& p);
gcn_status launch_gemm_rows(const GemmParams& p, void* ws, hipStream_t s);
// Weights split once for several row-panel products (gcn_epoch: the weights do not change
// between the forward and the backward pass).  A job is identified by the operand B as a
// product sees it: pointer, pitch, transposition and the k x n shape.
struct SplitJob {
  const float* B;
  int64_t ldb;
  bool tb;
  int64_t k, n;
  void* out;  // gemm_rows_split_bytes(job) bytes, 16-byte aligned
};
constexpr int kMaxSplitJobs = 16;
size_t gemm_rows_split_bytes(const SplitJob& j);
gcn_status launch_split_batch(const SplitJob* jobs, int count, hipStream_t s);
// The prepared planes for p's B, if any job matches it and p takes the row-panel kernel.
inline GemmParams with_split(GemmParams p, const SplitJob* jobs, int count) {
  if (!jobs || !gemm_rows_supported(p)) return p;
  for (int i = 0; i < count; ++i)
    if (jobs[i].B == p.B && jobs[i].ldb == p.ldb && jobs[i].tb == p.tb && jobs[i].k == p.k && jobs[i].n == p.n) {
      p.bsplit = jobs[i].out;
      break;
    }
  return p;
}
// Arithmetic of the dense products: bf16x6 (default) unless GCN_GEMM_MODE=fp32.
bool gemm_bf16x6_mode();
gcn_status launch_gemm(const GemmParams& p, void* ws, hipStream_t s);

size_t colsum_workspace(int64_t rows, int32_t w);
gcn_status launch_colsum(int64_t rows, int32_t w, const float* G, int64_t ldg, float* out,
                         const float* row_vals, float* mean, void* ws, hipStream_t s);

// exclusive scan of int32 counts into int64 offsets out[0..n], out[n] = total
size_t scan_workspace(int64_t n);
gcn_status launch_scan_i32(const int32_t* in, int64_t n, int64_t* out, void* ws, hipStream_t s);

size_t build_csr_workspace(int32_t n, int64_t n_edges);
gcn_status run_build_csr(int32_t n, int64_t n_edges, const int32_t* src, const int32_t* dst,
                         gcn_graph* g, void* ws, hipStream_t s);

size_t feature_stats_workspace(int32_t n, int32_t f, bool want_csc);
gcn_status run_feature_stats(const float* X, int32_t n, int32_t f, int64_t ldx, int32_t tau_num,
                             int32_t tau_den, int32_t force_mode, int64_t* row_nnz,
                             gcn_feature_info* info, gcn_sparse_x* x, void* ws, hipStream_t s);

// step >= 1 from the host, or (d_step != NULL) read from and incremented on the device
gcn_status launch_adam(const gcn_adam_tensor* t, int32_t count, int32_t step, int32_t* d_step, double lr,
                       double b1, double b2, double eps, hipStream_t s);

}  // namespace gcn
