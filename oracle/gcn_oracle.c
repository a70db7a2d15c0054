/*
 * gcn_oracle.c -- plain fp64 CPU oracle for the GCN training path (TEST
 * INFRASTRUCTURE ONLY).
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg load
 * this file's library.  The HIP library never includes, links or calls it,
 * and this file includes nothing from the HIP library.
 *
 * Each function is the plain definition of one step, written as straight
 * loops: no blocking, no fusion, no reordering beyond what the definition
 * states.  OpenMP only splits independent output rows over threads; every
 * output element is still produced by one sequential loop.  Floating point is
 * fp64 throughout; fp32 inputs are widened exactly.
 *
 * Paper: "Morphling: Fast, Fused, and Flexible GNN Training at Scale"
 * (arXiv 2512.01678).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_E_RANGE (-2)
#define ORC_E_CAPACITY (-4)
#define ORC_E_NOMEM (-7)

static int cmp_i32(const void* a, const void* b) {
  int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
  return (x > y) - (x < y);
}

/*
 * Graph of the GCN layer (Section III-A; the GCN of Kipf and Welling that the
 * paper cites for "normalized mean aggregation").  The neighbour set of node i
 * is the set of distinct j != i joined to i by an input edge in either
 * direction, plus i itself (the self-loop of A + I).  Input self pairs are
 * dropped before the one self-loop is added; repeated pairs count once.
 *
 * Output: row_ptr[n+1] (int64), col_idx[nnz] ascending within each row,
 * deg[i] = |row i| and dinv[i] = (float)(1 / sqrt((double)deg[i])).
 * Returns nnz, or ORC_E_RANGE if an id is outside [0, n), or ORC_E_CAPACITY
 * if nnz exceeds cap.
 */
int64_t orc_build_csr(int32_t n, int64_t n_edges, const int32_t* src, const int32_t* dst,
                      int64_t cap, int64_t* row_ptr, int32_t* col_idx, int32_t* deg,
                      float* dinv) {
  for (int64_t e = 0; e < n_edges; ++e)
    if (src[e] < 0 || src[e] >= n || dst[e] < 0 || dst[e] >= n) return ORC_E_RANGE;

  /* raw neighbour lists: both directions of every non-self edge, plus i itself */
  int64_t* start = (int64_t*)calloc((size_t)n + 1, sizeof(int64_t));
  int64_t* fill = (int64_t*)calloc((size_t)n + 1, sizeof(int64_t));
  if (!start || !fill) { free(start); free(fill); return ORC_E_NOMEM; }
  for (int32_t i = 0; i < n; ++i) start[i + 1] = 1;
  for (int64_t e = 0; e < n_edges; ++e) {
    if (src[e] == dst[e]) continue;
    start[src[e] + 1] += 1;
    start[dst[e] + 1] += 1;
  }
  for (int32_t i = 0; i < n; ++i) start[i + 1] += start[i];
  int32_t* raw = (int32_t*)malloc(sizeof(int32_t) * (size_t)(start[n] > 0 ? start[n] : 1));
  if (!raw) { free(start); free(fill); return ORC_E_NOMEM; }
  for (int32_t i = 0; i < n; ++i) { raw[start[i]] = i; fill[i] = start[i] + 1; }
  for (int64_t e = 0; e < n_edges; ++e) {
    int32_t u = src[e], v = dst[e];
    if (u == v) continue;
    raw[fill[u]++] = v;
    raw[fill[v]++] = u;
  }

  /* each row as a sorted set */
  int64_t total = 0;
  for (int32_t i = 0; i < n; ++i) {
    int32_t* r = raw + start[i];
    int64_t len = start[i + 1] - start[i];
    qsort(r, (size_t)len, sizeof(int32_t), cmp_i32);
    int64_t k = 0;
    for (int64_t t = 0; t < len; ++t)
      if (t == 0 || r[t] != r[t - 1]) r[k++] = r[t];
    deg[i] = (int32_t)k;
    total += k;
  }
  if (total > cap) { free(raw); free(start); free(fill); return ORC_E_CAPACITY; }
  row_ptr[0] = 0;
  for (int32_t i = 0; i < n; ++i) {
    row_ptr[i + 1] = row_ptr[i] + deg[i];
    memcpy(col_idx + row_ptr[i], raw + start[i], sizeof(int32_t) * (size_t)deg[i]);
    dinv[i] = (float)(1.0 / sqrt((double)deg[i]));
  }
  free(raw); free(start); free(fill);
  return total;
}

/*
 * Feature statistics (Section IV-B, "Sparsity Decision Model"; Algorithm 1,
 * Initialize): nnz(X) counts entries that compare unequal to 0.0f (so -0.0
 * is a zero and NaN a nonzero), per row and in total, as exact integers.
 */
int64_t orc_feature_counts(const float* X, int32_t n, int32_t f, int64_t ldx, int64_t* row_nnz) {
  int64_t total = 0;
#pragma omp parallel for reduction(+ : total) schedule(static)
  for (int32_t i = 0; i < n; ++i) {
    int64_t c = 0;
    for (int32_t j = 0; j < f; ++j)
      if (X[(int64_t)i * ldx + j] != 0.0f) c += 1;
    if (row_nnz) row_nnz[i] = c;
    total += c;
  }
  return total;
}

/*
 * Path decision (Section IV-B; Algorithm 1): the sparse path is taken when
 * s = 1 - nnz/(N F) >= tau, tau = tau_num / tau_den.  Evaluated exactly in
 * integers as tau_den * (N F - nnz) >= tau_num * N F.  Returns 1 for sparse.
 */
int32_t orc_sparse_decision(int64_t nnz, int64_t n, int64_t f, int32_t tau_num, int32_t tau_den) {
  __int128 nf = (__int128)n * f;
  __int128 lhs = (__int128)tau_den * (nf - nnz);
  __int128 rhs = (__int128)tau_num * nf;
  return lhs >= rhs ? 1 : 0;
}

/* DenseToCSR (Algorithm 1): row i lists (j, X_ij) for every nonzero, j ascending. */
void orc_dense_to_csr(const float* X, int32_t n, int32_t f, int64_t ldx, int64_t* row_ptr,
                      int32_t* col, float* val) {
  int64_t k = 0;
  row_ptr[0] = 0;
  for (int32_t i = 0; i < n; ++i) {
    for (int32_t j = 0; j < f; ++j) {
      float x = X[(int64_t)i * ldx + j];
      if (x != 0.0f) { col[k] = j; val[k] = x; ++k; }
    }
    row_ptr[i + 1] = k;
  }
}

/* DenseToCSC (Algorithm 1): column j lists (i, X_ij) for every nonzero, i ascending. */
void orc_dense_to_csc(const float* X, int32_t n, int32_t f, int64_t ldx, int64_t* col_ptr,
                      int32_t* row, float* val) {
  int64_t k = 0;
  col_ptr[0] = 0;
  for (int32_t j = 0; j < f; ++j) {
    for (int32_t i = 0; i < n; ++i) {
      float x = X[(int64_t)i * ldx + j];
      if (x != 0.0f) { row[k] = i; val[k] = x; ++k; }
    }
    col_ptr[j + 1] = k;
  }
}

/*
 * Linear aggregation Z = S M + 1 b^T over the rows of A + I (Section III-A, the
 * AGGREGATE step of a GNN layer; Algorithm 3 computes Y[u] = sum_e val[e] X[col[e]]
 * over the CSR row of u).  The operator S by `kind`:
 *   0  GCN normalised mean aggregation: S_uv = 1 / sqrt(d_u d_v)  (D^-1/2 (A+I) D^-1/2)
 *   1  sum aggregation (GIN with epsilon = 0): S_uv = 1             (A + I)
 *   2  mean aggregation: S_uv = 1 / d_u                             (D^-1 (A + I))
 *   3  transpose of the mean: S_uv = 1 / d_v                        ((A + I) D^-1)
 *
 * Rows listed in `rows` (all rows when rows == NULL) are written to Z at row
 * index r (the listed position when rows != NULL).  mag, when non-NULL, gets
 * sum |S_uv| |M_vc| + |b_c|, the magnitude scale of each output element.
 */
static double orc_weight(int32_t kind, int32_t du, int32_t dv) {
  switch (kind) {
    case 1: return 1.0;
    case 2: return 1.0 / (double)du;
    case 3: return 1.0 / (double)dv;
    default: return 1.0 / sqrt((double)du * (double)dv);
  }
}

void orc_aggregate(int32_t n, const int64_t* row_ptr, const int32_t* col_idx, const int32_t* deg,
                   const double* M, int64_t ldm, int32_t w, const double* bias, double* Z,
                   int64_t ldz, double* mag, const int32_t* rows, int64_t nrows, int32_t kind) {
  int64_t count = rows ? nrows : n;
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t r = 0; r < count; ++r) {
    int32_t u = rows ? rows[r] : (int32_t)r;
    double* z = Z + r * ldz;
    double* m = mag ? mag + r * ldz : NULL;
    for (int32_t c = 0; c < w; ++c) {
      z[c] = 0.0;
      if (m) m[c] = 0.0;
    }
    for (int64_t e = row_ptr[u]; e < row_ptr[u + 1]; ++e) {
      int32_t v = col_idx[e];
      double a = orc_weight(kind, deg[u], deg[v]);
      const double* mv = M + (int64_t)v * ldm;
      for (int32_t c = 0; c < w; ++c) {
        z[c] += a * mv[c];
        if (m) m[c] += a * fabs(mv[c]);
      }
    }
    if (bias)
      for (int32_t c = 0; c < w; ++c) {
        z[c] += bias[c];
        if (m) m[c] += fabs(bias[c]);
      }
  }
}

/*
 * Sparse-times-dense product with stored values: C[i,:] = sum_e val[e] B[idx[e],:]
 * over the compressed row i.  With X_csr this is the sparse forward X W
 * (Section IV-B, "Forward"); with X_csc (the CSR of X^T) it is the weight
 * gradient X^T G of the sparse backward (Algorithm 1, Backward).
 */
void orc_spmm(int64_t nrows, const int64_t* ptr, const int32_t* idx, const double* val,
              const double* B, int64_t ldb, int32_t w, double* C, int64_t ldc, double* mag) {
#pragma omp parallel for schedule(dynamic, 64)
  for (int64_t i = 0; i < nrows; ++i) {
    double* c = C + i * ldc;
    double* m = mag ? mag + i * ldc : NULL;
    for (int32_t k = 0; k < w; ++k) {
      c[k] = 0.0;
      if (m) m[k] = 0.0;
    }
    for (int64_t e = ptr[i]; e < ptr[i + 1]; ++e) {
      const double* b = B + (int64_t)idx[e] * ldb;
      for (int32_t k = 0; k < w; ++k) {
        c[k] += val[e] * b[k];
        if (m) m[k] += fabs(val[e] * b[k]);
      }
    }
  }
}

/*
 * Max aggregation (the "Max" aggregator of Listing 1; Section III-A lists mean,
 * max and sum): P[u,c] = max over the row of A + I of M[v,c], and argmax[u,c] =
 * the first v (columns ascending) that attains it.
 */
void orc_aggregate_max(int32_t n, const int64_t* row_ptr, const int32_t* col_idx, const double* M,
                       int64_t ldm, int32_t w, double* P, int32_t* argmax) {
#pragma omp parallel for schedule(dynamic, 64)
  for (int32_t u = 0; u < n; ++u) {
    for (int32_t c = 0; c < w; ++c) {
      double best = 0.0;
      int32_t arg = -1;
      for (int64_t e = row_ptr[u]; e < row_ptr[u + 1]; ++e) {
        int32_t v = col_idx[e];
        double x = M[(int64_t)v * ldm + c];
        if (arg < 0 || x > best) {
          best = x;
          arg = v;
        }
      }
      P[(int64_t)u * w + c] = best;
      argmax[(int64_t)u * w + c] = arg;
    }
  }
}

/*
 * Gradient of the max aggregation: each output element passes its gradient to the
 * one input it copied, dM[argmax[u,c], c] += dP[u,c] (every other input gets 0).
 * Written as that scatter, in row order, on one thread.
 */
void orc_aggregate_max_backward(int32_t n, const double* dP, int32_t w, const int32_t* argmax,
                                double* dM, int64_t ldo) {
  for (int32_t u = 0; u < n; ++u)
    for (int32_t c = 0; c < w; ++c) dM[(int64_t)u * ldo + c] = 0.0;
  for (int32_t u = 0; u < n; ++u)
    for (int32_t c = 0; c < w; ++c) dM[(int64_t)argmax[(int64_t)u * w + c] * ldo + c] += dP[(int64_t)u * w + c];
}
