// split.hip -- row-split plans for the long rows of a compressed matrix.
//
// A row with more than GCN_SPLIT_MIN entries is cut into GCN_SPLIT_CHUNK-entry
// chunks (see gcn_split in gcn.h).  Built once, during the blocking setup calls:
// per-row flags and chunk counts, two scans, one fill.  Rows are listed in
// ascending order and chunks row by row, so the plan is deterministic.  The
// optional processing order lists chunk k of every long row before chunk k+1 of
// any; for the CSC view of X, whose columns have similar densities, chunk k of
// every column then covers about the same window of rows, which stays in cache
// while all columns visit it.
#include <vector>

#include "internal.h"

namespace gcn {
namespace {

struct SplitWs {
  int32_t* is_long;
  int32_t* nch;
  int64_t* lidx;
  int64_t* choff;
  void* scan;
};

SplitWs carve(Arena& a, int64_t nrows) {
  SplitWs w;
  w.is_long = a.take<int32_t>(nrows);
  w.nch = a.take<int32_t>(nrows);
  w.lidx = a.take<int64_t>(nrows + 1);
  w.choff = a.take<int64_t>(nrows + 1);
  w.scan = a.take<char>((int64_t)scan_workspace(nrows + 1));
  return w;
}

__global__ void k_split_count(const int64_t* ptr, int64_t nrows, int32_t* is_long, int32_t* nch) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= nrows) return;
  const int64_t len = ptr[r + 1] - ptr[r];
  const bool lg = len > GCN_SPLIT_MIN;
  is_long[r] = lg ? 1 : 0;
  nch[r] = lg ? (int32_t)((len + GCN_SPLIT_CHUNK - 1) / GCN_SPLIT_CHUNK) : 0;
}

__global__ void k_split_fill(int64_t nrows, const int32_t* is_long, const int32_t* nch, const int64_t* lidx,
                             const int64_t* choff, int32_t* rows, int64_t* first, int32_t* owner) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r == 0) first[lidx[nrows]] = choff[nrows];
  if (r >= nrows || !is_long[r]) return;
  const int64_t h = lidx[r];
  rows[h] = (int32_t)r;
  first[h] = choff[r];
  for (int32_t k = 0; k < nch[r]; ++k) owner[choff[r] + k] = (int32_t)h;
}

}  // namespace

size_t split_workspace(int64_t nrows) {
  Arena a;
  carve(a, nrows);
  return a.used;
}

gcn_status build_split(const int64_t* ptr, int64_t nrows, gcn_split* sp, bool chunk_major, void* ws,
                       hipStream_t s) {
  sp->n_long = 0;
  sp->n_chunk = 0;
  if (nrows == 0) return GCN_OK;
  Arena a;
  a.base = static_cast<char*>(ws);
  SplitWs w = carve(a, nrows);
  const unsigned grid = (unsigned)ceil_div(nrows, 256);
  hipLaunchKernelGGL(k_split_count, dim3(grid), dim3(256), 0, s, ptr, nrows, w.is_long, w.nch);
  GCN_TRY(check_launch("split count"));
  GCN_TRY(launch_scan_i32(w.is_long, nrows, w.lidx, w.scan, s));
  GCN_TRY(launch_scan_i32(w.nch, nrows, w.choff, w.scan, s));
  int64_t tot[2];
  GCN_HIP(hipMemcpyAsync(&tot[0], w.lidx + nrows, sizeof(int64_t), hipMemcpyDeviceToHost, s), "split totals");
  GCN_HIP(hipMemcpyAsync(&tot[1], w.choff + nrows, sizeof(int64_t), hipMemcpyDeviceToHost, s), "split totals");
  GCN_HIP(hipStreamSynchronize(s), "split sync");
  if (tot[0] > sp->cap || tot[1] > sp->cap)
    return fail(GCN_E_CAPACITY, "split plan needs " + std::to_string(std::max(tot[0], tot[1])) +
                                    " entries, capacity " + std::to_string(sp->cap));
  if (tot[0] > INT32_MAX) return fail(GCN_E_OVERFLOW, "split plan: too many long rows");
  if (tot[0] > 0 || nrows > 0) {
    hipLaunchKernelGGL(k_split_fill, dim3(grid), dim3(256), 0, s, nrows, w.is_long, w.nch, w.lidx, w.choff,
                       sp->rows, sp->first, sp->owner);
    GCN_TRY(check_launch("split fill"));
  }
  sp->n_long = (int32_t)tot[0];
  sp->n_chunk = tot[1];
  if (chunk_major && sp->order && sp->n_chunk > 0) {
    std::vector<int64_t> first((size_t)sp->n_long + 1);
    GCN_HIP(hipMemcpyAsync(first.data(), sp->first, sizeof(int64_t) * first.size(), hipMemcpyDeviceToHost, s),
            "split first");
    GCN_HIP(hipStreamSynchronize(s), "split sync");
    std::vector<int64_t> order;
    order.reserve((size_t)sp->n_chunk);
    int64_t kmax = 0;
    for (int32_t h = 0; h < sp->n_long; ++h) kmax = std::max(kmax, first[h + 1] - first[h]);
    for (int64_t k = 0; k < kmax; ++k)
      for (int32_t h = 0; h < sp->n_long; ++h)
        if (first[h] + k < first[h + 1]) order.push_back(first[h] + k);
    GCN_HIP(hipMemcpyAsync(sp->order, order.data(), sizeof(int64_t) * order.size(), hipMemcpyHostToDevice, s),
            "split order");
    GCN_HIP(hipStreamSynchronize(s), "split sync");
  }
  return GCN_OK;
}

}  // namespace gcn
