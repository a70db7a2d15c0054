// fused.hip -- aggregate-first layer forward in one kernel (Section III-A's
// normalised aggregation followed by the dense transform of Algorithm 1):
//   P = A_hat X          (kept: the backward pass needs dW = P^T G)
//   H = act(P W + b)
// A workgroup owns a block of kRows rows.  Its eight wavefronts aggregate the rows
// with the same lane-slice code and slice count as the standalone aggregation (so P
// is bit-identical to it), prefetching each next row's offsets and first index chunk
// during the current row's gathers; they write each P row to memory and split it
// into three bf16 planes in LDS (the bf16x6 arithmetic of the dense products).  The
// block's rows then meet W on the matrix cores: every wavefront owns 32 output
// columns of each 256-column chunk, reads its A fragments from LDS and its W
// fragments (one step ahead) from planes of W that are split once per call and stay
// in L2, and applies bias and activation on the accumulators.  The aggregated block
// never goes back through HBM, and one workgroup's matrix-core phase overlaps the
// gathers of the others.
//
// Rows longer than the split threshold are summed by the chunk kernels of the
// standalone aggregation beforehand (their P rows are already in memory); the
// fused kernel reads those rows back instead of aggregating them.
#include "agg_device.h"
#include "bf16x6.h"

namespace gcn {
namespace {

constexpr int kRows = 64;  // rows per workgroup: two 32-row matrix-core tiles (measured
                           // faster than one: W fragments are fetched once per 64 rows)
constexpr int kWaves = 8;  // wavefronts per workgroup (measured: 5 % faster than 4, the
                           // LDS-bound workgroup count then holds more waves per CU)
constexpr int kThreads = 64 * kWaves;
constexpr int kColsPerWave = 256 / kWaves;  // output columns a wavefront owns per 256-column chunk

// W (k_in x n, row pitch ldw) -> three bf16 planes [3][n][kp], k-contiguous, zero
// for k >= k_in.  One thread per (column, pair of k).
__global__ void __launch_bounds__(256) k_split_w(const float* W, int64_t ldw, int32_t kin, int32_t n,
                                                 int32_t kp, uint32_t* planes) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t pairs = kp / 2;
  if (idx >= (int64_t)n * pairs) return;
  const int64_t col = idx / pairs;
  const int32_t k = (int32_t)(idx % pairs) * 2;
  const float a = k < kin ? W[(int64_t)k * ldw + col] : 0.f;
  const float b = k + 1 < kin ? W[(int64_t)(k + 1) * ldw + col] : 0.f;
  uint32_t hi, mid, lo;
  split_pair(a, b, hi, mid, lo);
  const int64_t plane = (int64_t)n * pairs;  // dwords per plane
  planes[idx] = hi;
  planes[plane + idx] = mid;
  planes[2 * plane + idx] = lo;
}

struct FusedArgs {
  AggParams a;          // rows, graph, X (M, ldm, w = f_in) and P (Z, ldz)
  const __bf16* wp;     // W planes [3][f_out][kp]
  int32_t kp, f_out;
  const float* bias;    // f_out or NULL
  float* H;
  int64_t ldh;
  int32_t relu;
  int32_t slots;        // neighbour slices per row (the standalone aggregation's choice)
  int64_t skip_over;    // rows longer than this already hold their P row
};

// KR rows per workgroup (KR / 32 matrix-core tiles along m), four wavefronts.
template <int LANES, int KR>
__global__ void __launch_bounds__(kThreads) k_agg_gemm(FusedArgs f) {
  constexpr int TM = KR / 32;
  constexpr int PITCH = LANES * 4 + 8;  // bf16 per plane row (a multiple of 8)
  constexpr int PLANE = KR * PITCH;
  __shared__ __attribute__((aligned(16))) __bf16 lds[3 * PLANE];
  const AggParams& p = f.a;
  const int wave = threadIdx.x / 64;
  const Lanes L = lanes_of<LANES, 4>(f.slots);  // blockIdx.y == 0: c0 = 4 * lane
  const int groups = 64 / L.gw;                 // rows a wavefront aggregates at a time
  const int grp = (threadIdx.x % 64) / L.gw;
  const int64_t r0 = (int64_t)blockIdx.x * KR;
  const bool cok = L.c0 < p.w;
  const bool cfull = L.c0 + 4 <= p.w;
  const int iters = KR / (kWaves * groups);
  auto row_of = [&](int it) { return r0 + (int64_t)(it * kWaves + wave) * groups + grp; };

  // ---- aggregation.  Two-stage prefetch along the wavefront's rows: the offsets of row
  // it + 2 and the first index chunk of row it + 1 are requested before the gathers of
  // row it, so the chain row offsets -> indices -> neighbour rows overlaps across rows.
  int64_t b1 = 0, e1 = 0, b2 = 0, e2 = 0;
  First f1{0, 0.f};
  {
    const int64_t ra = row_of(0);
    if (ra < p.n) {
      b1 = p.row_ptr[ra];
      e1 = p.row_ptr[ra + 1];
    }
    f1 = load_first<LANES>(p, b1, e1, L);
    const int64_t rb = iters > 1 ? row_of(1) : p.n;
    if (rb < p.n) {
      b2 = p.row_ptr[rb];
      e2 = p.row_ptr[rb + 1];
    }
  }
  for (int it = 0; it < iters; ++it) {
    const int64_t row = row_of(it);
    const int64_t beg = b1, end = e1;
    const First first = f1;
    b1 = b2;
    e1 = e2;
    f1 = load_first<LANES>(p, b1, e1, L);
    b2 = e2 = 0;
    const int64_t rn = it + 2 < iters ? row_of(it + 2) : p.n;
    if (rn < p.n) {
      b2 = p.row_ptr[rn];
      e2 = p.row_ptr[rn + 1];
    }
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (row < p.n) {
      float* prow = p.Z + row * p.ldz + L.c0;
      if (end - beg > f.skip_over) {
        if (cok) {
          if (cfull) {
            acc = *reinterpret_cast<const float4*>(prow);
          } else {
            acc.x = prow[0];
            if (L.c0 + 1 < p.w) acc.y = prow[1];
            if (L.c0 + 2 < p.w) acc.z = prow[2];
          }
        }
      } else {
        acc = accumulate<LANES, 4>(p, beg, end, L, f.slots, cok, first);
        const float sc = row_scale(p, row);
        acc.x *= sc;
        acc.y *= sc;
        acc.z *= sc;
        acc.w *= sc;
        if (cok && L.slot == 0) {
          if (cfull) {
            *reinterpret_cast<float4*>(prow) = acc;
          } else {
            prow[0] = acc.x;
            if (L.c0 + 1 < p.w) prow[1] = acc.y;
            if (L.c0 + 2 < p.w) prow[2] = acc.z;
          }
        }
      }
    }
    if (L.slot == 0) {
      // columns past f_in (and rows past n) enter the planes as zeros
      const float v0 = L.c0 + 0 < p.w ? acc.x : 0.f, v1 = L.c0 + 1 < p.w ? acc.y : 0.f;
      const float v2 = L.c0 + 2 < p.w ? acc.z : 0.f, v3 = L.c0 + 3 < p.w ? acc.w : 0.f;
      uint2 hi, mid, lo;
      split_pair(v0, v1, hi.x, mid.x, lo.x);
      split_pair(v2, v3, hi.y, mid.y, lo.y);
      __bf16* d = lds + (row - r0) * PITCH + L.c0;
      *reinterpret_cast<uint2*>(d) = hi;
      *reinterpret_cast<uint2*>(d + PLANE) = mid;
      *reinterpret_cast<uint2*>(d + 2 * PLANE) = lo;
    }
  }
  __syncthreads();

  // ---- transform: wavefront w owns columns 64 w .. 64 w + 63 of each 256-column chunk,
  // one 32-column tile at a time
  const int lane = threadIdx.x % 64;
  const int h = lane / 32, l32 = lane % 32;
  const int ksteps = f.kp / 16;
  const int64_t wplane = (int64_t)f.f_out * f.kp;
  const bool full_rows = r0 + KR <= p.n;
  for (int64_t n0 = (int64_t)wave * kColsPerWave; n0 < f.f_out; n0 += 256) {
#pragma unroll
    for (int j = 0; j < kColsPerWave / 32; ++j) {
      const int64_t col = n0 + j * 32 + l32;
      if (n0 + j * 32 >= f.f_out) break;  // wave-uniform
      // columns past f_out are computed from the last one and never stored
      const __bf16* wcol = f.wp + (col < f.f_out ? col : f.f_out - 1) * f.kp + h * 8;
      floatx16 acc[TM];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
      bf16x8 bh = *reinterpret_cast<const bf16x8*>(wcol);
      bf16x8 bm = *reinterpret_cast<const bf16x8*>(wcol + wplane);
      bf16x8 bl = *reinterpret_cast<const bf16x8*>(wcol + 2 * wplane);
      for (int ks = 0; ks < ksteps; ++ks) {
        const bf16x8 ch = bh, cm = bm, cl = bl;
        if (ks + 1 < ksteps) {  // next step's W fragments, from L2
          const __bf16* w = wcol + (ks + 1) * 16;
          bh = *reinterpret_cast<const bf16x8*>(w);
          bm = *reinterpret_cast<const bf16x8*>(w + wplane);
          bl = *reinterpret_cast<const bf16x8*>(w + 2 * wplane);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const __bf16* a = lds + (i * 32 + l32) * PITCH + ks * 16 + h * 8;
          const bf16x8 ah = *reinterpret_cast<const bf16x8*>(a);
          const bf16x8 am = *reinterpret_cast<const bf16x8*>(a + PLANE);
          const bf16x8 al = *reinterpret_cast<const bf16x8*>(a + 2 * PLANE);
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, ch, acc[i], 0, 0, 0);
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am, cm, acc[i], 0, 0, 0);
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, cl, acc[i], 0, 0, 0);
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am, ch, acc[i], 0, 0, 0);
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, cm, acc[i], 0, 0, 0);
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, ch, acc[i], 0, 0, 0);
        }
      }
      // lane l32 holds column l32 of the tile; register r holds row 8 (r / 4) + 4 h + r % 4
      if (col < f.f_out) {
        const float bj = f.bias ? f.bias[col] : 0.f;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          float* out = f.H + (r0 + i * 32 + 4 * h) * f.ldh + col;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int dr = 8 * (r / 4) + (r % 4);
            float v = acc[i][r] + bj;
            if (f.relu) v = fmaxf(v, 0.f);
            if (full_rows || r0 + i * 32 + 4 * h + dr < p.n) out[dr * f.ldh] = v;
          }
        }
      }
    }
  }
}

}  // namespace

bool agg_gemm_supported(int32_t f_in, int64_t ldx, int64_t ldp, const float* X, const float* P) {
  return f_in > 32 && f_in <= 128 && ldx % 4 == 0 && ldp % 4 == 0 && aligned16(X) && aligned16(P);
}

size_t agg_gemm_workspace(const gcn_split* split, int32_t f_in, int32_t f_out) {
  const int64_t kp = round_up(f_in, 16);
  return (size_t)round_up(6 * (int64_t)f_out * kp, 256) + aggregate_workspace(split, f_in);
}

gcn_status launch_agg_gemm(const AggParams& a, int64_t nnz, const gcn_split* split, const float* W,
                           int64_t ldw, int32_t f_out, const float* bias, bool relu, float* H, int64_t ldh,
                           void* ws, hipStream_t s) {
  if (a.n == 0 || f_out == 0) return GCN_OK;
  const int32_t kp = (int32_t)round_up(a.w, 16);
  char* w = static_cast<char*>(ws);
  uint32_t* planes = reinterpret_cast<uint32_t*>(w);
  void* aws = w + round_up(6 * (int64_t)f_out * kp, 256);
  char name[64];
  snprintf(name, sizeof name, "agg_gemm_%dx%d", a.w, f_out);
  ProfScope prof(name, f_out, a.n, nnz, s);
  const int64_t pairs = (int64_t)f_out * (kp / 2);
  hipLaunchKernelGGL(k_split_w, dim3((unsigned)ceil_div(pairs, 256)), dim3(256), 0, s, W, ldw, a.w, f_out, kp,
                     planes);
  GCN_TRY(check_launch("split W"));
  // long rows: the standalone chunk kernels write their P rows first
  const bool split_rows = has_split(split);
  if (split_rows) GCN_TRY(launch_aggregate_long_rows(a, split, aws, s));
  FusedArgs f;
  f.a = a;
  f.wp = reinterpret_cast<const __bf16*>(planes);
  f.kp = kp;
  f.f_out = f_out;
  f.bias = bias;
  f.H = H;
  f.ldh = ldh;
  f.relu = relu ? 1 : 0;
  f.skip_over = split_rows ? (int64_t)GCN_SPLIT_MIN : INT64_MAX;
  const dim3 grid((unsigned)ceil_div(a.n, kRows));
  if (a.w <= 64) {
    f.slots = agg_slots(16, nnz, a.n);
    hipLaunchKernelGGL((k_agg_gemm<16, kRows>), grid, dim3(kThreads), 0, s, f);
  } else {
    f.slots = agg_slots(32, nnz, a.n);
    hipLaunchKernelGGL((k_agg_gemm<32, kRows>), grid, dim3(kThreads), 0, s, f);
  }
  return check_launch("aggregate-transform");
}

}  // namespace gcn
