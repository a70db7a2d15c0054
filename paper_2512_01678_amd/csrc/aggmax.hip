// aggmax.hip -- max aggregation over the rows of A + I and its gradient.
//
// Section III-A names mean, max and sum aggregators; Listing 1 trains GraphSAGE
// with "Max".  Forward, per row u and column c:
//   P[u,c] = max over v in row u of M[v,c],  arg[u,c] = the first such v
// (columns ascending), the same lane-slice mapping as the linear aggregation:
// each slice keeps (value, column) of its entries in order, and slices combine by
// "larger value, then smaller column", so the result does not depend on how the
// row was cut.  Backward is the gradient's gather form over the symmetric rows:
//   dM[u,c] = sum over v in row u of dP[v,c] * [arg[v,c] == u]
// (optionally times 1[mask > 0]); no atomics, fixed order.  Rows are not split
// into chunks here: a long row is walked by one lane group.
#include "agg_device.h"

namespace gcn {
namespace {

constexpr int kBlock = 256;

struct MaxArgs {
  AggParams a;          // rows / graph and M (forward) or dP (backward) in a.M, a.ldm
  int32_t* arg;         // forward output
  const int32_t* carg;  // backward input
  int64_t ldarg;
  float* out;           // P (forward) or dM (backward)
  int64_t ldo;
  const float* mask;    // backward: 1[mask > 0] applied when non-NULL
  int64_t ldmask;
};

template <int VEC>
struct Lane {
  float v[VEC];
  int j[VEC];
};

template <int LANES, int VEC>
__global__ void __launch_bounds__(kBlock) k_agg_max(MaxArgs m, int slots) {
  using V = Vec<VEC>;
  constexpr int UNR = LANES >= 4 ? 8 : 4;
  const AggParams& p = m.a;
  const Lanes L = lanes_of<LANES, VEC>(slots);
  const int64_t row = (int64_t)blockIdx.x * (kBlock / L.gw) + threadIdx.x / L.gw;
  if (row >= p.n) return;  // whole groups leave together
  const int64_t beg = p.row_ptr[row], end = p.row_ptr[row + 1];
  const bool cok = L.c0 < p.w;
  Lane<VEC> best;
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    best.v[i] = -INFINITY;
    best.j[i] = INT32_MAX;
  }
  const float* Mc = p.M + L.c0;
  for (int64_t base = beg; base < end; base += L.gw) {
    const int cnt = (int)((end - base) < L.gw ? (end - base) : L.gw);
    const int my_j = L.lig < cnt ? p.col[base + L.lig] : 0;
    for (int t = 0; t < cnt; t += slots * UNR) {
      int jj[UNR];
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
      for (int u = 0; u < UNR; ++u) {
        if (!ok[u]) continue;
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
          const float x = V::get(xs[u], i);
          // entries of a slice come in increasing column order: strict > keeps the first
          if (x > best.v[i] || best.j[i] == INT32_MAX) {
            best.v[i] = x;
            best.j[i] = jj[u];
          }
        }
      }
    }
  }
  // combine the slices: larger value, then smaller column
  for (int o = LANES; o < L.gw; o <<= 1) {
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      const float ov = __shfl_xor(best.v[i], o, L.gw);
      const int oj = __shfl_xor(best.j[i], o, L.gw);
      if (ov > best.v[i] || (ov == best.v[i] && oj < best.j[i]) || best.j[i] == INT32_MAX) {
        if (oj != INT32_MAX) {
          best.v[i] = ov;
          best.j[i] = oj;
        }
      }
    }
  }
  if (!cok || L.slot != 0) return;
  float* po = m.out + row * m.ldo + L.c0;
  int32_t* ao = m.arg + row * m.ldarg + L.c0;
#pragma unroll
  for (int i = 0; i < VEC; ++i)
    if (L.c0 + i < p.w) {
      po[i] = best.v[i];
      ao[i] = best.j[i];
    }
}

template <int LANES, int VEC, bool MASK>
__global__ void __launch_bounds__(kBlock) k_agg_max_bwd(MaxArgs m, int slots) {
  using V = Vec<VEC>;
  constexpr int UNR = LANES >= 4 ? 8 : 4;
  const AggParams& p = m.a;
  const Lanes L = lanes_of<LANES, VEC>(slots);
  const int64_t row = (int64_t)blockIdx.x * (kBlock / L.gw) + threadIdx.x / L.gw;
  if (row >= p.n) return;
  const int64_t beg = p.row_ptr[row], end = p.row_ptr[row + 1];
  const bool cok = L.c0 < p.w;
  float acc[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) acc[i] = 0.f;
  const float* Dc = p.M + L.c0;
  const int32_t* Ac = m.carg + L.c0;
  const int me = (int)row;
  for (int64_t base = beg; base < end; base += L.gw) {
    const int cnt = (int)((end - base) < L.gw ? (end - base) : L.gw);
    const int my_j = L.lig < cnt ? p.col[base + L.lig] : 0;
    for (int t = 0; t < cnt; t += slots * UNR) {
      int jj[UNR];
      bool ok[UNR];
      typename V::T xs[UNR];
      int as[UNR][VEC];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int e = t + u * slots + L.slot;
        ok[u] = e < cnt;
        jj[u] = __shfl(my_j, ok[u] ? e : 0, L.gw);
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        xs[u] = V::zero();
#pragma unroll
        for (int i = 0; i < VEC; ++i) as[u][i] = -1;
        if (ok[u] && cok) {
          xs[u] = V::load(Dc + (int64_t)jj[u] * p.ldm);
          const int32_t* ap = Ac + (int64_t)jj[u] * m.ldarg;
          if constexpr (VEC == 4) {
            const int4 a4 = *reinterpret_cast<const int4*>(ap);
            as[u][0] = a4.x;
            as[u][VEC > 1 ? 1 : 0] = a4.y;
            as[u][VEC > 2 ? 2 : 0] = a4.z;
            as[u][VEC > 3 ? 3 : 0] = a4.w;
          } else {
            as[u][0] = ap[0];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u)
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] += as[u][i] == me ? V::get(xs[u], i) : 0.f;
    }
  }
  for (int o = LANES; o < L.gw; o <<= 1)
#pragma unroll
    for (int i = 0; i < VEC; ++i) acc[i] += __shfl_xor(acc[i], o, L.gw);
  if (!cok || L.slot != 0) return;
  float* out = m.out + row * m.ldo + L.c0;
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    if (L.c0 + i >= p.w) continue;
    float v = acc[i];
    if constexpr (MASK) v = m.mask[row * m.ldmask + L.c0 + i] > 0.f ? v : 0.f;
    out[i] = v;
  }
}

template <int VEC, class F>
gcn_status dispatch_lanes(int lanes, F&& f) {
  switch (lanes) {
    case 1: return f(std::integral_constant<int, 1>{});
    case 2: return f(std::integral_constant<int, 2>{});
    case 4: return f(std::integral_constant<int, 4>{});
    case 8: return f(std::integral_constant<int, 8>{});
    case 16: return f(std::integral_constant<int, 16>{});
    case 32: return f(std::integral_constant<int, 32>{});
    default: return f(std::integral_constant<int, 64>{});
  }
}

}  // namespace

// vec4 needs 16-byte rows for every operand the kernel touches
static bool max_vec4(const MaxArgs& m, bool fwd) {
  const AggParams& p = m.a;
  bool ok = p.ldm % 4 == 0 && aligned16(p.M) && m.ldo % 4 == 0 && aligned16(m.out) && m.ldarg % 4 == 0;
  ok = ok && aligned16(fwd ? (const void*)m.arg : (const void*)m.carg);
  if (!fwd && m.mask) ok = ok && m.ldmask % 4 == 0 && aligned16(m.mask);
  return ok;
}

static gcn_status launch_max(const MaxArgs& m, int64_t nnz, bool fwd, hipStream_t s) {
  const AggParams& p = m.a;
  if (p.n == 0 || p.w == 0) return GCN_OK;
  const bool vec4 = max_vec4(m, fwd);
  const int vec = vec4 ? 4 : 1;
  int lanes = 1;
  while (lanes < ceil_div(p.w, vec) && lanes < 64) lanes <<= 1;
  if ((int64_t)lanes * vec < p.w) return fail(GCN_E_UNSUPPORTED, "max aggregation: width above 256 (vector) or 64");
  const int slots = agg_slots(lanes, nnz, p.n);
  const int gw = lanes * slots;
  const dim3 grid((unsigned)ceil_div(p.n, kBlock / gw));
  char name[64];
  snprintf(name, sizeof name, "%s_w%d", fwd ? "aggmax" : "aggmax_bwd", p.w);
  ProfScope prof(name, p.w, p.n, nnz, s);
  auto go = [&](auto lt) -> gcn_status {
    constexpr int LN = decltype(lt)::value;
    if (vec4) {
      if (fwd) hipLaunchKernelGGL((k_agg_max<LN, 4>), grid, dim3(kBlock), 0, s, m, slots);
      else if (m.mask) hipLaunchKernelGGL((k_agg_max_bwd<LN, 4, true>), grid, dim3(kBlock), 0, s, m, slots);
      else hipLaunchKernelGGL((k_agg_max_bwd<LN, 4, false>), grid, dim3(kBlock), 0, s, m, slots);
    } else {
      if (fwd) hipLaunchKernelGGL((k_agg_max<LN, 1>), grid, dim3(kBlock), 0, s, m, slots);
      else if (m.mask) hipLaunchKernelGGL((k_agg_max_bwd<LN, 1, true>), grid, dim3(kBlock), 0, s, m, slots);
      else hipLaunchKernelGGL((k_agg_max_bwd<LN, 1, false>), grid, dim3(kBlock), 0, s, m, slots);
    }
    return check_launch(fwd ? "max aggregation" : "max aggregation gradient");
  };
  return vec4 ? dispatch_lanes<4>(lanes, go) : dispatch_lanes<1>(lanes, go);
}

gcn_status launch_aggregate_max(const AggParams& p, int64_t nnz, float* P, int64_t ldp, int32_t* arg,
                                int64_t ldarg, hipStream_t s) {
  MaxArgs m{};
  m.a = p;
  m.arg = arg;
  m.ldarg = ldarg;
  m.out = P;
  m.ldo = ldp;
  return launch_max(m, nnz, true, s);
}

gcn_status launch_aggregate_max_bwd(const AggParams& p, int64_t nnz, const int32_t* arg, int64_t ldarg,
                                    const float* mask, int64_t ldmask, float* dM, int64_t ldo, hipStream_t s) {
  MaxArgs m{};
  m.a = p;
  m.carg = arg;
  m.ldarg = ldarg;
  m.out = dM;
  m.ldo = ldo;
  m.mask = mask;
  m.ldmask = ldmask;
  return launch_max(m, nnz, false, s);
}

}  // namespace gcn
