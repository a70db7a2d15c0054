// agg_device.h -- device-side building blocks of the row-parallel sparse products
// (included by the aggregation kernels and the fused aggregate-then-transform kernel).
//
// A slice of LANES lanes covers a row's columns, VEC consecutive columns per lane;
// `slots` slices share a row and take every slots-th entry; UNR neighbour-row loads
// are kept in flight per lane; the slices are summed with cross-lane adds, so every
// slice ends with the row's total.  No atomics: results are deterministic.
#pragma once

#include "internal.h"
#include "lanes.h"

#ifndef GCN_AGG_UNR
#define GCN_AGG_UNR 16  // neighbour-row loads kept in flight per lane, full-wavefront rows
#endif

namespace gcn {
namespace {

template <int VEC>
struct Vec;
template <>
struct Vec<4> {
  using T = float4;
  static __device__ __forceinline__ T load(const float* p) { return *reinterpret_cast<const float4*>(p); }
  static __device__ __forceinline__ void store(float* p, const T& v) { *reinterpret_cast<float4*>(p) = v; }
  static __device__ __forceinline__ T zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
  static __device__ __forceinline__ void fma(T& acc, float w, const T& x) {
    acc.x = fmaf(w, x.x, acc.x);
    acc.y = fmaf(w, x.y, acc.y);
    acc.z = fmaf(w, x.z, acc.z);
    acc.w = fmaf(w, x.w, acc.w);
  }
  static __device__ __forceinline__ void add(T& acc, const T& x) {
    acc.x += x.x;
    acc.y += x.y;
    acc.z += x.z;
    acc.w += x.w;
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
  static __device__ __forceinline__ void store(float* p, const T& v) { *p = v; }
  static __device__ __forceinline__ T zero() { return 0.f; }
  static __device__ __forceinline__ void fma(T& acc, float w, const T& x) { acc = fmaf(w, x, acc); }
  static __device__ __forceinline__ void add(T& acc, const T& x) { acc += x; }
  static __device__ __forceinline__ float get(const T& v, int) { return v; }
  static __device__ __forceinline__ void add_xor(T& v, int o, int width) { v += __shfl_xor(v, o, width); }
};

template <int LANES>
__device__ __forceinline__ float group_max(float v) {
  return group_reduce<LANES>(v, [](float a, float b) { return fmaxf(a, b); });
}
template <int LANES>
__device__ __forceinline__ float group_sum(float v) {
  return group_reduce<LANES>(v, [](float a, float b) { return a + b; });
}

// Lane geometry of a group of LANES * slots lanes owning one (virtual) row.
struct Lanes {
  int gw, lig, slot, lane, c0;
};

template <int LANES, int VEC>
__device__ __forceinline__ Lanes lanes_of(int slots) {
  Lanes L;
  L.gw = LANES * slots;
  L.lig = threadIdx.x & (L.gw - 1);
  L.slot = L.lig / LANES;
  L.lane = L.lig & (LANES - 1);
  L.c0 = (blockIdx.y * LANES + L.lane) * VEC;
  return L;
}

// Column index and value of entry beg + lig (lane lig of the group), the first chunk
// of a row; zero past the row's end.
struct First {
  int j;
  float w;
};

// Weight of entry e (column j) by the aggregation kind (wave-uniform branch).
__device__ __forceinline__ float entry_weight(const AggParams& p, int64_t e, int j) {
  if (p.kind == AGG_W_VAL) return p.val[e];
  if (p.kind == AGG_W_COLMEAN) return 1.f / (float)p.deg[j];
  return 1.f;
}

// Factor applied to a row's sum: 1 / deg[row] for the mean, else 1.
__device__ __forceinline__ float row_scale(const AggParams& p, int64_t row) {
  return p.kind == AGG_W_ROWMEAN ? 1.f / (float)p.deg[row] : 1.f;
}

template <int LANES>
__device__ __forceinline__ First load_first(const AggParams& p, int64_t beg, int64_t end, const Lanes& L) {
  First f{0, 0.f};
  if (beg + L.lig < end) {
    f.j = p.col[beg + L.lig];
    f.w = entry_weight(p, beg + L.lig, f.j);
  }
  return f;
}

// sum_{e in [beg, end)} w_e M[col[e], c0 .. c0+VEC), every slice of the group holding the
// total.  first: the group's first chunk of entries (load_first), already requested by
// the caller.
template <int LANES, int VEC>
__device__ __forceinline__ typename Vec<VEC>::T accumulate(const AggParams& p, int64_t beg, int64_t end,
                                                           const Lanes& L, int slots, bool cok, First first) {
  using V = Vec<VEC>;
  constexpr int UNR = LANES == 64 ? GCN_AGG_UNR : (LANES >= 4 ? 8 : 4);
  typename V::T acc = V::zero();
  const float* Mc = p.M + L.c0;
  for (int64_t base = beg; base < end; base += L.gw) {
    const int cnt = (int)((end - base) < L.gw ? (end - base) : L.gw);
    int my_j = first.j;
    float my_w = first.w;
    if (base != beg) {
      my_j = L.lig < cnt ? p.col[base + L.lig] : 0;
      my_w = L.lig < cnt ? entry_weight(p, base + L.lig, my_j) : 0.f;
    }
    for (int t = 0; t < cnt; t += slots * UNR) {
      int jj[UNR];
      float ww[UNR];
      bool ok[UNR];
      typename V::T xs[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = t + u * slots + L.slot;
        ok[u] = e < cnt;
        jj[u] = __shfl(my_j, ok[u] ? e : 0, L.gw);
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) xs[u] = (ok[u] && cok) ? V::load(Mc + (int64_t)jj[u] * p.ldm) : V::zero();
#pragma unroll
      for (int u = 0; u < UNR; ++u) ww[u] = __shfl(my_w, ok[u] ? t + u * slots + L.slot : 0, L.gw);
#pragma unroll
      for (int u = 0; u < UNR; ++u) V::fma(acc, ok[u] ? ww[u] : 0.f, xs[u]);
    }
  }
  for (int o = LANES; o < L.gw; o <<= 1) V::add_xor(acc, o, L.gw);
  return acc;
}


}  // namespace
}  // namespace gcn
