// features.hip -- density probe and compressed views of the input features.
//
// Section IV-B / Algorithm 1 (Initialize): s = 1 - nnz(X)/(N F) is measured
// once at load time; the sparse path is taken iff s >= tau, and then X is
// converted to CSR (forward) and CSC (backward).  Everything here is integer
// work (counts, offsets, index lists) plus bit-exact copies of the values, so
// the results are identical to any other correct construction.
//
//  * per-row counts: one wavefront per row, columns 64 at a time;
//  * DenseToCSR: the same walk, each nonzero placed by the popcount of the
//    wavefront's ballot below its lane (columns stay ascending);
//  * DenseToCSC: rows are cut into chunks; per (chunk, column) counts, a
//    per-column scan over chunks, then each chunk writes its entries of every
//    column at that column's offset while walking its rows in order, so rows
//    stay ascending within a column without any sort.
#include "internal.h"

namespace gcn {
namespace {

constexpr int kChunkRows = 1024;

struct FeatWs {
  int32_t* row_cnt;    // n
  int64_t* row_off;    // n + 1 (used when the caller supplies no CSR buffer)
  void* scan;
  int32_t* chunk_cnt;  // nchunks * f
  int32_t* chunk_off;  // nchunks * f
  int32_t* col_tot;    // f
  int64_t nchunks;
  void* split;         // split plan scratch for long CSC columns
};

FeatWs carve(Arena& a, int32_t n, int32_t f, bool csc) {
  FeatWs w;
  w.row_cnt = a.take<int32_t>(n);
  w.row_off = a.take<int64_t>((int64_t)n + 1);
  w.scan = a.take<char>((int64_t)scan_workspace(std::max<int64_t>(n, f) + 1));
  w.nchunks = ceil_div(n, kChunkRows);
  w.chunk_cnt = a.take<int32_t>(csc ? w.nchunks * f : 0);
  w.chunk_off = a.take<int32_t>(csc ? w.nchunks * f : 0);
  w.col_tot = a.take<int32_t>(csc ? f : 0);
  w.split = a.take<char>(csc ? (int64_t)split_workspace(f) : 0);
  return w;
}

__global__ void __launch_bounds__(256) k_row_counts(const float* X, int32_t n, int32_t f, int64_t ldx,
                                                    int32_t* cnt, int64_t* cnt64) {
  const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / 64;
  const int lane = threadIdx.x % 64;
  if (row >= n) return;
  const float* x = X + row * ldx;
  int c = 0;
  for (int j = lane; j < f; j += 64) c += x[j] != 0.0f ? 1 : 0;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
  if (lane == 0) {
    cnt[row] = c;
    if (cnt64) cnt64[row] = c;
  }
}

__global__ void __launch_bounds__(256) k_to_csr(const float* X, int32_t n, int32_t f, int64_t ldx,
                                                const int64_t* row_ptr, int32_t* col, float* val) {
  const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / 64;
  const int lane = threadIdx.x % 64;
  if (row >= n) return;
  const float* x = X + row * ldx;
  int64_t pos = row_ptr[row];
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int j0 = 0; j0 < f; j0 += 64) {
    const int j = j0 + lane;
    const float v = j < f ? x[j] : 0.0f;
    const bool nz = v != 0.0f;
    const uint64_t bal = __ballot(nz);
    if (nz) {
      const int64_t p = pos + __popcll(bal & below);
      col[p] = j;
      val[p] = v;
    }
    pos += __popcll(bal);
  }
}

// counts of nonzeros per (row chunk, column)
__global__ void __launch_bounds__(256) k_chunk_counts(const float* X, int32_t n, int32_t f, int64_t ldx,
                                                      int32_t* chunk_cnt) {
  const int64_t r0 = (int64_t)blockIdx.x * kChunkRows;
  const int64_t r1 = std::min<int64_t>(r0 + kChunkRows, n);
  for (int j = threadIdx.x; j < f; j += blockDim.x) {
    int c = 0;
    for (int64_t r = r0; r < r1; ++r) c += X[r * ldx + j] != 0.0f ? 1 : 0;
    chunk_cnt[blockIdx.x * (int64_t)f + j] = c;
  }
}

// per column: exclusive offsets of each chunk within the column, and the column total
__global__ void k_chunk_scan(int64_t nchunks, int32_t f, const int32_t* chunk_cnt, int32_t* chunk_off,
                             int32_t* col_tot) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= f) return;
  int32_t run = 0;
  for (int64_t c = 0; c < nchunks; ++c) {
    chunk_off[c * f + j] = run;
    run += chunk_cnt[c * f + j];
  }
  col_tot[j] = run;
}

__global__ void __launch_bounds__(256) k_to_csc(const float* X, int32_t n, int32_t f, int64_t ldx,
                                                const int64_t* col_ptr, const int32_t* chunk_off,
                                                int32_t* rowi, float* val) {
  const int64_t r0 = (int64_t)blockIdx.x * kChunkRows;
  const int64_t r1 = std::min<int64_t>(r0 + kChunkRows, n);
  for (int j = threadIdx.x; j < f; j += blockDim.x) {
    int64_t pos = col_ptr[j] + chunk_off[blockIdx.x * (int64_t)f + j];
    for (int64_t r = r0; r < r1; ++r) {
      const float v = X[r * ldx + j];
      if (v != 0.0f) {
        rowi[pos] = (int32_t)r;
        val[pos] = v;
        ++pos;
      }
    }
  }
}

}  // namespace

size_t feature_stats_workspace(int32_t n, int32_t f, bool want_csc) {
  Arena a;
  carve(a, n, f, want_csc);
  return a.used;
}

gcn_status run_feature_stats(const float* X, int32_t n, int32_t f, int64_t ldx, int32_t tau_num,
                             int32_t tau_den, int32_t force_mode, int64_t* row_nnz,
                             gcn_feature_info* info, gcn_sparse_x* x, void* ws, hipStream_t s) {
  const bool want_csc = x && x->col_ptr;
  Arena a;
  a.base = static_cast<char*>(ws);
  FeatWs w = carve(a, n, f, want_csc);
  const unsigned gw = (unsigned)std::max<int64_t>(1, ceil_div(n, 4));
  if (n > 0) {
    hipLaunchKernelGGL(k_row_counts, dim3(gw), dim3(256), 0, s, X, n, f, ldx, w.row_cnt, row_nnz);
    GCN_TRY(check_launch("feature row counts"));
  }
  int64_t* rp = (x && x->row_ptr) ? x->row_ptr : w.row_off;
  GCN_TRY(launch_scan_i32(w.row_cnt, n, rp, w.scan, s));
  int64_t nnz = 0;
  GCN_HIP(hipMemcpyAsync(&nnz, rp + n, sizeof nnz, hipMemcpyDeviceToHost, s), "feature nnz");
  GCN_HIP(hipStreamSynchronize(s), "feature sync");
  const __int128 nf = (__int128)n * f;
  info->nnz = nnz;
  info->sparsity = nf > 0 ? 1.0 - (double)nnz / (double)nf : 0.0;
  const bool sparse = (__int128)tau_den * (nf - nnz) >= (__int128)tau_num * nf;
  info->mode = force_mode >= 0 ? force_mode : (sparse ? GCN_SPARSE : GCN_DENSE);
  if (!x) return GCN_OK;

  if (nnz > x->nnz)
    return fail(GCN_E_CAPACITY, "gcn_feature_stats: nnz(X) = " + std::to_string(nnz) +
                                    " exceeds the sparse capacity " + std::to_string(x->nnz));
  x->nnz = nnz;
  x->n = n;
  x->f = f;
  if (n > 0) {
    hipLaunchKernelGGL(k_to_csr, dim3(gw), dim3(256), 0, s, X, n, f, ldx, x->row_ptr, x->col, x->val);
    GCN_TRY(check_launch("dense to csr"));
  }
  if (want_csc) {
    if (w.nchunks > 0) {
      hipLaunchKernelGGL(k_chunk_counts, dim3((unsigned)w.nchunks), dim3(256), 0, s, X, n, f, ldx,
                         w.chunk_cnt);
      GCN_TRY(check_launch("csc chunk counts"));
    }
    hipLaunchKernelGGL(k_chunk_scan, dim3((unsigned)std::max<int64_t>(1, ceil_div(f, 256))), dim3(256),
                       0, s, w.nchunks, f, w.chunk_cnt, w.chunk_off, w.col_tot);
    GCN_TRY(check_launch("csc chunk scan"));
    GCN_TRY(launch_scan_i32(w.col_tot, f, x->col_ptr, w.scan, s));
    if (w.nchunks > 0) {
      hipLaunchKernelGGL(k_to_csc, dim3((unsigned)w.nchunks), dim3(256), 0, s, X, n, f, ldx, x->col_ptr,
                         w.chunk_off, x->row, x->cval);
      GCN_TRY(check_launch("dense to csc"));
    }
    if (x->csc_split.rows) GCN_TRY(build_split(x->col_ptr, f, &x->csc_split, true, w.split, s));
  }
  GCN_HIP(hipStreamSynchronize(s), "feature sync");
  return GCN_OK;
}

}  // namespace gcn
