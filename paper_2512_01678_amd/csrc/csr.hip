// csr.hip -- A + I in CSR form from an edge list, on the device.
//
// Section III-A's GCN operator needs, for every node, the set of its distinct
// neighbours plus itself, in a fixed (ascending) order so that the result is
// canonical and bit-exact against any other correct construction.
//
//  1. count: every non-self input pair adds one raw entry to both endpoint rows;
//     each row starts with its self entry (integer atomics: counts only).
//  2. scan the raw counts into raw row offsets.
//  3. fill: scatter both directions of each pair into the raw rows (the order
//     within a row depends on scheduling; step 4 removes that dependence).
//  4. sort + deduplicate each raw row in place, by row length:
//       <= 64 entries    one wavefront, rank by cross-lane comparison;
//       <= 4096 entries  one workgroup, bitonic sort in LDS;
//       larger           one workgroup, a bitmap over all n columns in the
//                        workspace, read back in column order.
//  5. scan the unique counts (the degrees) into row_ptr; compact into col_idx
//     and write dinv = (float)(1 / sqrt((double)deg)).
//  6. write the entries of A_hat, val[e] = dinv[row] * dinv[col[e]] (fp32).
//  7. (optional) the row order of the aggregations: rows by decreasing length class,
//     longest first, so that the long rows start early and the short ones fill the end
//     of a launch (a longest-job-first schedule; the results do not depend on it).  A
//     stable counting sort over 64 classes of the degree: per-block class counts, one
//     scan in class-major order, then each block places its rows (ties in row order).
#include "internal.h"

namespace gcn {
namespace {

constexpr int kSmall = 64;
constexpr int kMedium = 4096;
constexpr int kLargeBlocks = 64;

struct CsrWs {
  int32_t* cnt;       // n: raw entries per row
  int32_t* fillc;     // n: fill cursors
  int64_t* raw_off;   // n + 1
  int32_t* raw;       // 2 E + n
  int32_t* lists;     // 3 n: small / medium / large row lists
  int32_t* flags;     // [0] range error, [1..3] list sizes
  void* scan;
  uint32_t* bitmap;   // kLargeBlocks * words
  int64_t words;
  void* split;        // hub split plan scratch
  int32_t* ord_cnt;   // kClasses * blocks of 256 rows: rows per (class, block)
  int64_t* ord_off;   // kClasses * blocks + 1: their exclusive scan
};

constexpr int kClasses = 64;
constexpr int kOrderBlock = 256;
inline int64_t order_blocks(int32_t n) { return ceil_div(n > 0 ? n : 1, kOrderBlock); }

CsrWs carve(Arena& a, int32_t n, int64_t n_edges) {
  CsrWs w;
  w.cnt = a.take<int32_t>(n);
  w.fillc = a.take<int32_t>(n);
  w.raw_off = a.take<int64_t>((int64_t)n + 1);
  w.raw = a.take<int32_t>(2 * n_edges + n);
  w.lists = a.take<int32_t>(3 * (int64_t)n);
  w.flags = a.take<int32_t>(8);
  const int64_t ocount = kClasses * order_blocks(n);
  w.scan = a.take<char>((int64_t)scan_workspace(std::max<int64_t>((int64_t)n + 1, ocount + 1)));
  w.words = ceil_div(n, 32);
  w.bitmap = a.take<uint32_t>(kLargeBlocks * w.words);
  w.split = a.take<char>((int64_t)split_workspace(n));
  w.ord_cnt = a.take<int32_t>(ocount);
  w.ord_off = a.take<int64_t>(ocount + 1);
  return w;
}

__global__ void k_init(int32_t n, int32_t* cnt, int32_t* fillc, int32_t* flags) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    cnt[i] = 1;
    fillc[i] = 1;
  }
  if (i < 8) flags[i] = 0;
}

__global__ void k_count(int32_t n, int64_t ne, const int32_t* src, const int32_t* dst, int32_t* cnt,
                        int32_t* flags) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < ne;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int32_t u = src[e], v = dst[e];
    if (u < 0 || u >= n || v < 0 || v >= n) {
      atomicOr(&flags[0], 1);
      continue;
    }
    if (u == v) continue;
    atomicAdd(&cnt[u], 1);
    atomicAdd(&cnt[v], 1);
  }
}

__global__ void k_fill(int32_t n, int64_t ne, const int32_t* src, const int32_t* dst,
                       const int64_t* off, int32_t* fillc, int32_t* raw) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = t0; i < n; i += stride) raw[off[i]] = (int32_t)i;
  for (int64_t e = t0; e < ne; e += stride) {
    const int32_t u = src[e], v = dst[e];
    if (u == v) continue;
    raw[off[u] + atomicAdd(&fillc[u], 1)] = v;
    raw[off[v] + atomicAdd(&fillc[v], 1)] = u;
  }
}

// Row lists by length class; one atomic per class per wavefront (ballot-aggregated).
__global__ void __launch_bounds__(256) k_classify(int32_t n, const int32_t* cnt, int32_t* lists, int32_t* flags) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int lane = threadIdx.x % 64;
  int cls = -1;
  if (i < n) {
    const int32_t len = cnt[i];
    cls = len <= kSmall ? 0 : (len <= kMedium ? 1 : 2);
  }
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  for (int c = 0; c < 3; ++c) {
    const uint64_t bal = __ballot(cls == c);
    if (!bal) continue;
    const int leader = __ffsll((unsigned long long)bal) - 1;
    int32_t base = 0;
    if (lane == leader) base = atomicAdd(&flags[1 + c], (int32_t)__popcll(bal));
    base = __shfl(base, leader);
    if (cls == c) lists[(int64_t)c * n + base + (int32_t)__popcll(bal & below)] = (int32_t)i;
  }
}

// one wavefront per row of <= 64 entries
__global__ void __launch_bounds__(256) k_sort_small(int32_t count, const int32_t* list,
                                                    const int64_t* off, const int32_t* cnt,
                                                    int32_t* raw, int32_t* deg) {
  const int64_t wid = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / 64;
  const int lane = threadIdx.x % 64;
  if (wid >= count) return;
  const int32_t row = list[wid];
  const int32_t len = cnt[row];
  int32_t* seg = raw + off[row];
  const int32_t x = lane < len ? seg[lane] : INT32_MAX;
  bool first = lane < len;
  for (int k = 0; k < 64; ++k) {
    const int32_t xk = __shfl(x, k);
    if (k < lane && xk == x) first = false;
  }
  int rank = 0;
  for (int k = 0; k < 64; ++k) {
    const int32_t xk = __shfl(x, k);
    const int fk = __shfl((int)first, k);
    if (fk && xk < x) ++rank;
  }
  const uint64_t bal = __ballot(first);
  if (first) seg[rank] = x;
  if (lane == 0) deg[row] = (int32_t)__popcll(bal);
}

// one workgroup per row of 65..4096 entries: bitonic sort in LDS, then compact
__global__ void __launch_bounds__(256) k_sort_medium(int32_t count, const int32_t* list,
                                                     const int64_t* off, const int32_t* cnt,
                                                     int32_t* raw, int32_t* deg) {
  __shared__ int32_t a[kMedium];
  __shared__ int32_t part[256];
  const int tid = threadIdx.x;
  for (int64_t item = blockIdx.x; item < count; item += gridDim.x) {
    const int32_t row = list[item];
    const int32_t len = cnt[row];
    int32_t* seg = raw + off[row];
    int P = 256;
    while (P < len) P <<= 1;
    for (int i = tid; i < P; i += 256) a[i] = i < len ? seg[i] : INT32_MAX;
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1) {
      for (int j = k >> 1; j > 0; j >>= 1) {
        for (int i = tid; i < P; i += 256) {
          const int ij = i ^ j;
          if (ij > i) {
            const int32_t x = a[i], y = a[ij];
            const bool up = (i & k) == 0;
            if ((x > y) == up) {
              a[i] = y;
              a[ij] = x;
            }
          }
        }
        __syncthreads();
      }
    }
    // each thread owns P/256 consecutive slots
    const int per = P / 256;
    const int b0 = tid * per;
    int c = 0;
    for (int i = b0; i < b0 + per; ++i)
      if (i < len && (i == 0 || a[i] != a[i - 1])) ++c;
    part[tid] = c;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {
      const int add = tid >= o ? part[tid - o] : 0;
      __syncthreads();
      part[tid] += add;
      __syncthreads();
    }
    int pos = part[tid] - c;
    for (int i = b0; i < b0 + per; ++i)
      if (i < len && (i == 0 || a[i] != a[i - 1])) seg[pos++] = a[i];
    if (tid == 255) deg[row] = part[255];
    __syncthreads();
  }
}

// one workgroup per row of > 4096 entries: set bits in an n-bit map, read back in order.
// The map is touched only with device-scope atomics, so no stale cache line is read.
__global__ void __launch_bounds__(256) k_sort_large(int32_t count, const int32_t* list,
                                                    const int64_t* off, const int32_t* cnt,
                                                    int32_t* raw, int32_t* deg, uint32_t* bitmap,
                                                    int64_t words) {
  __shared__ int32_t part[256];
  const int tid = threadIdx.x;
  uint32_t* bm = bitmap + (int64_t)blockIdx.x * words;
  for (int64_t item = blockIdx.x; item < count; item += gridDim.x) {
    const int32_t row = list[item];
    const int32_t len = cnt[row];
    int32_t* seg = raw + off[row];
    for (int64_t w = tid; w < words; w += 256)
      __hip_atomic_store(&bm[w], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __threadfence();
    __syncthreads();
    for (int64_t j = tid; j < len; j += 256) {
      const int32_t x = seg[j];
      atomicOr(&bm[x >> 5], 1u << (x & 31));
    }
    __threadfence();
    __syncthreads();
    int64_t run = 0;
    constexpr int kPer = 8;
    for (int64_t w0 = 0; w0 < words; w0 += 256 * kPer) {
      uint32_t v[kPer];
      int c = 0;
      for (int i = 0; i < kPer; ++i) {
        const int64_t w = w0 + (int64_t)tid * kPer + i;
        v[i] = w < words ? __hip_atomic_load(&bm[w], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0u;
        c += __popc(v[i]);
      }
      part[tid] = c;
      __syncthreads();
      for (int o = 1; o < 256; o <<= 1) {
        const int add = tid >= o ? part[tid - o] : 0;
        __syncthreads();
        part[tid] += add;
        __syncthreads();
      }
      int64_t pos = run + part[tid] - c;
      const int total = part[255];
      for (int i = 0; i < kPer; ++i) {
        uint32_t bits = v[i];
        const int64_t base = (w0 + (int64_t)tid * kPer + i) * 32;
        while (bits) {
          const int b = __ffs(bits) - 1;
          bits &= bits - 1;
          seg[pos++] = (int32_t)(base + b);
        }
      }
      run += total;
      __syncthreads();
    }
    if (tid == 0) deg[row] = (int32_t)run;
    __threadfence();
    __syncthreads();
  }
}

__global__ void __launch_bounds__(256) k_compact(int32_t n, const int64_t* raw_off, const int32_t* raw,
                                                 const int64_t* row_ptr, const int32_t* deg,
                                                 int32_t* col_idx, float* dinv) {
  const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / 64;
  const int lane = threadIdx.x % 64;
  if (row >= n) return;
  const int32_t d = deg[row];
  const int32_t* s = raw + raw_off[row];
  int32_t* o = col_idx + row_ptr[row];
  for (int32_t j = lane; j < d; j += 64) o[j] = s[j];
  if (lane == 0) dinv[row] = (float)(1.0 / sqrt((double)d));
}

__global__ void __launch_bounds__(256) k_values(int32_t n, const int64_t* row_ptr, const int32_t* col_idx,
                                                const float* dinv, float* val) {
  const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / 64;
  const int lane = threadIdx.x % 64;
  if (row >= n) return;
  const float di = dinv[row];
  for (int64_t e = row_ptr[row] + lane; e < row_ptr[row + 1]; e += 64) val[e] = di * dinv[col_idx[e]];
}

// Length class of a row: 4 classes per power of two of the degree (its two bits below
// the leading one), class 0 for the longest rows (degree >= 2^15.75).
__device__ __forceinline__ int length_class(int32_t d) {
  if (d < 4) return kClasses - 1 - d;
  const int lg = 31 - __clz(d);
  const int key = 4 * lg + ((d >> (lg - 2)) & 3);
  return kClasses - 1 - (key < kClasses - 1 ? key : kClasses - 1);
}

__global__ void __launch_bounds__(kOrderBlock) k_order_count(int32_t n, const int32_t* deg, int32_t* cnt,
                                                             int64_t nblk) {
  __shared__ int32_t h[kClasses];
  if (threadIdx.x < kClasses) h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t row = (int64_t)blockIdx.x * kOrderBlock + threadIdx.x;
  if (row < n) atomicAdd(&h[length_class(deg[row])], 1);  // LDS integer counts
  __syncthreads();
  if (threadIdx.x < kClasses) cnt[(int64_t)threadIdx.x * nblk + blockIdx.x] = h[threadIdx.x];
}

__global__ void __launch_bounds__(kOrderBlock) k_order_place(int32_t n, const int32_t* deg, const int64_t* off,
                                                             int64_t nblk, int32_t* order) {
  __shared__ int32_t cls[kOrderBlock];
  const int64_t row = (int64_t)blockIdx.x * kOrderBlock + threadIdx.x;
  const int c = row < n ? length_class(deg[row]) : -1;
  cls[threadIdx.x] = c;
  __syncthreads();
  if (row >= n) return;
  int rank = 0;  // rows of the same class before this one in the block
  for (int t = 0; t < (int)threadIdx.x; ++t) rank += cls[t] == c ? 1 : 0;
  order[off[(int64_t)c * nblk + blockIdx.x] + rank] = (int32_t)row;
}

}  // namespace

size_t build_csr_workspace(int32_t n, int64_t n_edges) {
  Arena a;
  carve(a, n, n_edges);
  return a.used;
}

gcn_status run_build_csr(int32_t n, int64_t n_edges, const int32_t* src, const int32_t* dst,
                         gcn_graph* g, void* ws, hipStream_t s) {
  Arena a;
  a.base = static_cast<char*>(ws);
  CsrWs w = carve(a, n, n_edges);
  const int T = 256;
  const unsigned gn = (unsigned)ceil_div(n > 8 ? n : 8, T);
  const unsigned ge = (unsigned)(ceil_div(n_edges, T) < 65536 ? (ceil_div(n_edges, T) > 0 ? ceil_div(n_edges, T) : 1) : 65536);

  hipLaunchKernelGGL(k_init, dim3(gn), dim3(T), 0, s, n, w.cnt, w.fillc, w.flags);
  GCN_TRY(check_launch("csr init"));
  hipLaunchKernelGGL(k_count, dim3(ge), dim3(T), 0, s, n, n_edges, src, dst, w.cnt, w.flags);
  GCN_TRY(check_launch("csr count"));
  int32_t flags[4];
  GCN_HIP(hipMemcpyAsync(flags, w.flags, sizeof flags, hipMemcpyDeviceToHost, s), "csr flags");
  GCN_HIP(hipStreamSynchronize(s), "csr sync");
  if (flags[0]) return fail(GCN_E_RANGE, "gcn_build_csr: an edge endpoint is outside [0, n)");

  GCN_TRY(launch_scan_i32(w.cnt, n, w.raw_off, w.scan, s));
  const unsigned gf = (unsigned)std::max<int64_t>(1, std::min<int64_t>(65536, ceil_div(std::max<int64_t>(n_edges, n), T)));
  hipLaunchKernelGGL(k_fill, dim3(gf), dim3(T), 0, s, n, n_edges, src, dst, w.raw_off, w.fillc, w.raw);
  GCN_TRY(check_launch("csr fill"));
  hipLaunchKernelGGL(k_classify, dim3(gn), dim3(T), 0, s, n, w.cnt, w.lists, w.flags);
  GCN_TRY(check_launch("csr classify"));
  GCN_HIP(hipMemcpyAsync(flags, w.flags, sizeof flags, hipMemcpyDeviceToHost, s), "csr flags");
  GCN_HIP(hipStreamSynchronize(s), "csr sync");
  const int32_t n_small = flags[1], n_med = flags[2], n_large = flags[3];
  if (n_small > 0) {
    hipLaunchKernelGGL(k_sort_small, dim3((unsigned)ceil_div(n_small, 4)), dim3(256), 0, s, n_small,
                       w.lists, w.raw_off, w.cnt, w.raw, g->deg);
    GCN_TRY(check_launch("csr sort small"));
  }
  if (n_med > 0) {
    const unsigned gm = (unsigned)std::min<int64_t>(n_med, 8192);
    hipLaunchKernelGGL(k_sort_medium, dim3(gm), dim3(256), 0, s, n_med, w.lists + n, w.raw_off,
                       w.cnt, w.raw, g->deg);
    GCN_TRY(check_launch("csr sort medium"));
  }
  if (n_large > 0) {
    const unsigned gl = (unsigned)std::min<int64_t>(n_large, kLargeBlocks);
    hipLaunchKernelGGL(k_sort_large, dim3(gl), dim3(256), 0, s, n_large, w.lists + 2 * (int64_t)n,
                       w.raw_off, w.cnt, w.raw, g->deg, w.bitmap, w.words);
    GCN_TRY(check_launch("csr sort large"));
  }
  GCN_TRY(launch_scan_i32(g->deg, n, g->row_ptr, w.scan, s));
  int64_t nnz = 0;
  GCN_HIP(hipMemcpyAsync(&nnz, g->row_ptr + n, sizeof nnz, hipMemcpyDeviceToHost, s), "csr nnz");
  GCN_HIP(hipStreamSynchronize(s), "csr sync");
  g->nnz = nnz;
  if (nnz > g->nnz_cap)
    return fail(GCN_E_CAPACITY, "gcn_build_csr: nnz " + std::to_string(nnz) + " exceeds nnz_cap " +
                                    std::to_string(g->nnz_cap));
  if (n > 0) {
    hipLaunchKernelGGL(k_compact, dim3((unsigned)ceil_div(n, 4)), dim3(256), 0, s, n, w.raw_off, w.raw,
                       g->row_ptr, g->deg, g->col_idx, g->dinv);
    GCN_TRY(check_launch("csr compact"));
    hipLaunchKernelGGL(k_values, dim3((unsigned)ceil_div(n, 4)), dim3(256), 0, s, n, g->row_ptr, g->col_idx,
                       g->dinv, g->val);
    GCN_TRY(check_launch("csr values"));
  }
  if (g->order && n > 0) {
    const int64_t nblk = order_blocks(n);
    hipLaunchKernelGGL(k_order_count, dim3((unsigned)nblk), dim3(kOrderBlock), 0, s, n, g->deg, w.ord_cnt, nblk);
    GCN_TRY(check_launch("csr order count"));
    GCN_TRY(launch_scan_i32(w.ord_cnt, kClasses * nblk, w.ord_off, w.scan, s));
    hipLaunchKernelGGL(k_order_place, dim3((unsigned)nblk), dim3(kOrderBlock), 0, s, n, g->deg, w.ord_off, nblk,
                       g->order);
    GCN_TRY(check_launch("csr order place"));
  }
  g->split.order = nullptr;
  if (g->split.rows) GCN_TRY(build_split(g->row_ptr, n, &g->split, false, w.split, s));
  GCN_HIP(hipStreamSynchronize(s), "csr sync");
  return GCN_OK;
}

}  // namespace gcn
