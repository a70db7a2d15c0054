// aggregate.hip -- row-parallel sparse aggregation on gfx950.
//
// Z[u,:] = s_u * sum_{e in row u} w_e * M[col[e], :]  (+ bias, epilogue)
//
//  * normalised GCN aggregation (Section III-A): w_e = dinv[col[e]], s_u = dinv[u],
//    so Z = A_hat M with A_hat = D^-1/2 (A + I) D^-1/2;
//  * sparse-feature products (Section IV-B): w_e = val[e], s_u = 1 (X_csr W, X_csc G).
//
// Mapping (the paper's row-per-block idea of Algorithm 3, re-cut for 64-wide
// wavefronts): a slice of LANES lanes covers the row's columns, each lane VEC
// consecutive columns, so one neighbour row is fetched as LANES coalesced
// 16-byte loads.  A row is owned by `slots` such slices (LANES * slots <= 64
// lanes); slice k takes neighbours k, k + slots, ...  The row's lanes read the
// column indices cooperatively (one per lane), broadcast each index and weight
// with a cross-lane shuffle, and keep UNR neighbour loads in flight before the
// FMAs.  The slices are summed with cross-lane adds at the end.  Accumulators
// stay in registers and every output element is written once, so no atomics
// are involved and results are deterministic.  Narrow rows of low-degree
// graphs pack several rows into one wavefront (slots = 1).
#include "internal.h"

namespace gcn {
namespace {

template <int VEC>
struct Vec;
template <>
struct Vec<4> {
  using T = float4;
  static __device__ __forceinline__ T load(const float* p) { return *reinterpret_cast<const float4*>(p); }
  static __device__ __forceinline__ T zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
  static __device__ __forceinline__ void fma(T& acc, float w, const T& x) {
    acc.x = fmaf(w, x.x, acc.x);
    acc.y = fmaf(w, x.y, acc.y);
    acc.z = fmaf(w, x.z, acc.z);
    acc.w = fmaf(w, x.w, acc.w);
  }
  static __device__ __forceinline__ float get(const T& v, int i) {
    return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
  }
  static __device__ __forceinline__ void add_xor(T& v, int o, int width) {
    v.x += __shfl_xor(v.x, o, width);
    v.y += __shfl_xor(v.y, o, width);
    v.z += __shfl_xor(v.z, o, width);
    v.w += __shfl_xor(v.w, o, width);
  }
};
template <>
struct Vec<1> {
  using T = float;
  static __device__ __forceinline__ T load(const float* p) { return *p; }
  static __device__ __forceinline__ T zero() { return 0.f; }
  static __device__ __forceinline__ void fma(T& acc, float w, const T& x) { acc = fmaf(w, x, acc); }
  static __device__ __forceinline__ float get(const T& v, int) { return v; }
  static __device__ __forceinline__ void add_xor(T& v, int o, int width) { v += __shfl_xor(v, o, width); }
};

template <int LANES>
__device__ __forceinline__ float group_max(float v) {
#pragma unroll
  for (int o = LANES / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, LANES));
  return v;
}
template <int LANES>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int o = LANES / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, LANES);
  return v;
}

constexpr int kBlock = 256;

// One row per group of LANES * slots lanes (slots is a power of two, LANES * slots <= 64).
// Each of the `slots` lane slices walks every slots-th neighbour of the row; the slices
// are summed at the end with cross-lane adds in a fixed pattern (deterministic).
template <int LANES, int VEC, int EPI, bool USE_VAL>
__global__ void __launch_bounds__(kBlock) k_aggregate(AggParams p, int slots) {
  using V = Vec<VEC>;
  constexpr int UNR = LANES >= 4 ? 8 : 4;
  const int gw = LANES * slots;
  const int lig = threadIdx.x & (gw - 1);
  const int slot = lig / LANES;
  const int lane = lig & (LANES - 1);
  const int64_t row = (int64_t)blockIdx.x * (kBlock / gw) + threadIdx.x / gw;
  const bool live = row < p.n;
  const int c0 = (blockIdx.y * LANES + lane) * VEC;
  const bool cok = live && c0 < p.w;

  int64_t beg = 0, end = 0;
  if (live) {
    beg = p.row_ptr[row];
    end = p.row_ptr[row + 1];
  }
  typename V::T acc = V::zero();
  const float* Mc = p.M + c0;
  for (int64_t base = beg; base < end; base += gw) {
    const int cnt = (int)((end - base) < gw ? (end - base) : gw);
    int my_j = 0;
    float my_w = 0.f;
    if (lig < cnt) {
      my_j = p.col[base + lig];
      my_w = USE_VAL ? p.val[base + lig] : p.dinv[my_j];
    }
    for (int t = 0; t < cnt; t += slots * UNR) {
      int jj[UNR];
      float ww[UNR];
      bool ok[UNR];
      typename V::T xs[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = t + u * slots + slot;
        ok[u] = e < cnt;
        const int src = ok[u] ? e : 0;
        jj[u] = __shfl(my_j, src, gw);
        ww[u] = __shfl(my_w, src, gw);
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) xs[u] = (ok[u] && cok) ? V::load(Mc + (int64_t)jj[u] * p.ldm) : V::zero();
#pragma unroll
      for (int u = 0; u < UNR; ++u) V::fma(acc, ok[u] ? ww[u] : 0.f, xs[u]);
    }
  }
  // sum the slices: after this every slice holds the full row
  for (int o = LANES; o < gw; o <<= 1) V::add_xor(acc, o, gw);
  if (!live) return;

  const float s = USE_VAL ? 1.f : p.dinv[row];
  float z[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    const int c = c0 + i;
    z[i] = s * V::get(acc, i);
    if (p.bias && c < p.w) z[i] += p.bias[c];
  }

  if constexpr (EPI == AGG_SOFTMAX) {
    // whole logits row is held by each slice (w <= LANES * VEC); slice 0 writes
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < VEC; ++i)
      if (c0 + i < p.w) mx = fmaxf(mx, z[i]);
    mx = group_max<LANES>(mx);
    float e[VEC];
    float se = 0.f;
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      e[i] = (c0 + i < p.w) ? expf(z[i] - mx) : 0.f;
      se += e[i];
    }
    se = group_sum<LANES>(se);
    const int y = p.labels[row];
    float zy = 0.f;
#pragma unroll
    for (int i = 0; i < VEC; ++i)
      if (c0 + i == y) zy = z[i];
    zy = group_sum<LANES>(zy);
    if (slot != 0) return;
    if (lane == 0) p.row_loss[row] = (logf(se) + mx) - zy;
    if (!cok) return;
    const float inv_se = 1.f / se;
    float gv[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) gv[i] = (e[i] * inv_se - (c0 + i == y ? 1.f : 0.f)) * p.inv_n;
    float* out = p.Z + row * p.ldz + c0;
    float* lg = p.logits ? p.logits + row * p.ldl + c0 : nullptr;
    if (VEC == 4 && c0 + 4 <= p.w) {
      *reinterpret_cast<float4*>(out) = make_float4(gv[0], gv[VEC > 1 ? 1 : 0], gv[VEC > 2 ? 2 : 0],
                                                    gv[VEC > 3 ? 3 : 0]);
    } else {
#pragma unroll
      for (int i = 0; i < VEC; ++i)
        if (c0 + i < p.w) out[i] = gv[i];
    }
    if (lg) {
#pragma unroll
      for (int i = 0; i < VEC; ++i)
        if (c0 + i < p.w) lg[i] = z[i];
    }
    return;
  } else {
    if (!cok || slot != 0) return;
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      if constexpr (EPI == AGG_RELU) z[i] = fmaxf(z[i], 0.f);
      if constexpr (EPI == AGG_MASK) {
        const int c = c0 + i;
        if (c < p.w) z[i] = p.mask[row * p.ldmask + c] > 0.f ? z[i] : 0.f;
      }
    }
    float* out = p.Z + row * p.ldz + c0;
    if (VEC == 4 && c0 + 4 <= p.w) {
      *reinterpret_cast<float4*>(out) = make_float4(z[0], z[VEC > 1 ? 1 : 0], z[VEC > 2 ? 2 : 0],
                                                    z[VEC > 3 ? 3 : 0]);
    } else {
#pragma unroll
      for (int i = 0; i < VEC; ++i)
        if (c0 + i < p.w) out[i] = z[i];
    }
  }
}

template <int LANES, int VEC, int EPI>
gcn_status launch3(const AggParams& p, int slots, hipStream_t s) {
  const int gw = LANES * slots;
  dim3 grid((unsigned)ceil_div(p.n, kBlock / gw), (unsigned)ceil_div(p.w, LANES * VEC));
  if constexpr (EPI == AGG_NONE) {
    if (p.val) {
      hipLaunchKernelGGL((k_aggregate<LANES, VEC, EPI, true>), grid, dim3(kBlock), 0, s, p, slots);
      return check_launch("spmm");
    }
  }
  hipLaunchKernelGGL((k_aggregate<LANES, VEC, EPI, false>), grid, dim3(kBlock), 0, s, p, slots);
  return check_launch("aggregate");
}

template <int LANES, int VEC>
gcn_status launch2(const AggParams& p, int slots, hipStream_t s) {
  switch (p.epi) {
    case AGG_NONE: return launch3<LANES, VEC, AGG_NONE>(p, slots, s);
    case AGG_RELU: return launch3<LANES, VEC, AGG_RELU>(p, slots, s);
    case AGG_MASK: return launch3<LANES, VEC, AGG_MASK>(p, slots, s);
    default: return launch3<LANES, VEC, AGG_SOFTMAX>(p, slots, s);
  }
}

template <int VEC>
gcn_status launch1(const AggParams& p, int lanes, int slots, hipStream_t s) {
  switch (lanes) {
    case 1: return launch2<1, VEC>(p, slots, s);
    case 2: return launch2<2, VEC>(p, slots, s);
    case 4: return launch2<4, VEC>(p, slots, s);
    case 8: return launch2<8, VEC>(p, slots, s);
    case 16: return launch2<16, VEC>(p, slots, s);
    case 32: return launch2<32, VEC>(p, slots, s);
    default: return launch2<64, VEC>(p, slots, s);
  }
}

// Neighbour slices per row: as many as keep at least 2 neighbours per slice on an
// average row (slices beyond that would mostly idle), within one wavefront.
int pick_slots(int lanes, int64_t nnz, int64_t rows) {
  const int max_slots = std::min(64 / lanes, 16);
  if (const char* e = getenv("GCN_AGG_SLOTS")) {
    int v = atoi(e), s = 1;
    while (s * 2 <= v && s * 2 <= max_slots) s *= 2;
    return s;
  }
  if (nnz < 0 || rows <= 0) return 1;
  const double avg = (double)nnz / (double)rows;
  int s = 1;
  while (s * 2 <= max_slots && 2.0 * (s * 2) <= avg) s *= 2;
  return s;
}

}  // namespace

gcn_status launch_aggregate(const AggParams& p, int64_t nnz, hipStream_t s) {
  if (p.n == 0 || p.w == 0) return GCN_OK;
  const bool vec4 = p.ldm % 4 == 0 && p.ldz % 4 == 0 && aligned16(p.M) && aligned16(p.Z) &&
                    (p.epi != AGG_MASK || (p.ldmask % 4 == 0 && aligned16(p.mask)));
  const int vec = vec4 ? 4 : 1;
  int need = (int)ceil_div(p.w, vec);
  int lanes = 1;
  while (lanes < need && lanes < 64) lanes <<= 1;
  if (p.epi == AGG_SOFTMAX && need > lanes)
    return fail(GCN_E_UNSUPPORTED, "softmax epilogue needs width <= 256 (vector) or 64 (scalar)");
  const int slots = pick_slots(lanes, nnz, p.n);
  char name[64];
  snprintf(name, sizeof name, "%s_w%d", p.val ? "spmm" : "aggregate", p.w);
  ProfScope prof(name, p.w, p.n, nnz, s);
  return vec4 ? launch1<4>(p, lanes, slots, s) : launch1<1>(p, lanes, slots, s);
}

}  // namespace gcn
