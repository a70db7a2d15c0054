// scan.hip -- exclusive prefix sum of int32 counts into int64 offsets.
//
// Three launches: per-tile sums, one workgroup scanning the tile sums, and a
// per-tile rescan that adds the tile's offset.  Integer arithmetic, so the
// result does not depend on scheduling.
#include "internal.h"

namespace gcn {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 8;
constexpr int kTile = kThreads * kItems;

__device__ int64_t block_exclusive_scan(int64_t v, int64_t* total) {
  __shared__ int64_t buf[kThreads];
  const int t = threadIdx.x;
  buf[t] = v;
  __syncthreads();
  for (int o = 1; o < kThreads; o <<= 1) {
    const int64_t add = t >= o ? buf[t - o] : 0;
    __syncthreads();
    buf[t] += add;
    __syncthreads();
  }
  const int64_t incl = buf[t];
  *total = buf[kThreads - 1];
  __syncthreads();
  return incl - v;
}

__global__ void __launch_bounds__(kThreads) k_tile_sums(const int32_t* in, int64_t n, int64_t* sums) {
  const int64_t base = (int64_t)blockIdx.x * kTile + threadIdx.x * kItems;
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kItems; ++i)
    if (base + i < n) s += in[base + i];
  int64_t total;
  block_exclusive_scan(s, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// one workgroup: sums[0..nt) -> exclusive offsets, out[n] = grand total
__global__ void __launch_bounds__(kThreads) k_scan_sums(int64_t* sums, int64_t nt, int64_t* out, int64_t n) {
  int64_t carry = 0;
  for (int64_t c0 = 0; c0 < nt; c0 += kThreads) {
    const int64_t i = c0 + threadIdx.x;
    const int64_t v = i < nt ? sums[i] : 0;
    int64_t total;
    const int64_t ex = block_exclusive_scan(v, &total);
    if (i < nt) sums[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) out[n] = carry;
}

__global__ void __launch_bounds__(kThreads) k_tile_apply(const int32_t* in, int64_t n, const int64_t* sums,
                                                         int64_t* out) {
  const int64_t base = (int64_t)blockIdx.x * kTile + threadIdx.x * kItems;
  int32_t v[kItems];
  int64_t s = 0;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    v[i] = base + i < n ? in[base + i] : 0;
    s += v[i];
  }
  int64_t total;
  int64_t run = block_exclusive_scan(s, &total) + sums[blockIdx.x];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
}

}  // namespace

size_t scan_workspace(int64_t n) { return sizeof(int64_t) * (size_t)(ceil_div(n, kTile) + 1); }

gcn_status launch_scan_i32(const int32_t* in, int64_t n, int64_t* out, void* ws, hipStream_t s) {
  const int64_t nt = ceil_div(n, kTile);
  int64_t* sums = static_cast<int64_t*>(ws);
  if (nt > 0) {
    hipLaunchKernelGGL(k_tile_sums, dim3((unsigned)nt), dim3(kThreads), 0, s, in, n, sums);
    GCN_TRY(check_launch("scan tile sums"));
  }
  hipLaunchKernelGGL(k_scan_sums, dim3(1), dim3(kThreads), 0, s, sums, nt, out, n);
  GCN_TRY(check_launch("scan sums"));
  if (nt > 0) {
    hipLaunchKernelGGL(k_tile_apply, dim3((unsigned)nt), dim3(kThreads), 0, s, in, n, sums, out);
    GCN_TRY(check_launch("scan apply"));
  }
  return GCN_OK;
}

}  // namespace gcn
