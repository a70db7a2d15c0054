// aggregate.hip -- row-parallel sparse aggregation on gfx950.
//
// Z[u,:] = sum_{e in row u} val[e] * M[col[e], :]  (+ bias, epilogue)
//
//  * normalised GCN aggregation (Section III-A): val holds the entries of
//    A_hat = D^-1/2 (A + I) D^-1/2, computed once when the graph is built;
//  * sparse-feature products (Section IV-B): X_csr W and X_csc G.
//
// Each entry's weight is read beside its column index: no per-entry gather of
// degree data sits between the index load and the neighbour-row gather.
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
//
// Long rows (hubs; more than GCN_SPLIT_MIN entries) would leave one group
// walking the whole row while the rest of the GPU idles.  With a split plan,
// the main kernel skips them; k_chunks sums each GCN_SPLIT_CHUNK-entry chunk
// into a partial row, and k_combine adds a long row's partials in chunk order
// and applies the same epilogue.
#include "agg_device.h"

#include <cstring>
#include <type_traits>

namespace gcn {
namespace {

constexpr int kBlock = 256;

// Bias and epilogue of one row.  Every slice of the group holds the row's total and
// slice 0 writes; with OWN, each slice holds a row of its own (own: that row exists and
// is finished here) and writes it.
template <int LANES, int VEC, int EPI, bool OWN = false>
__device__ __forceinline__ void finish_row(const AggParams& p, int64_t row, const typename Vec<VEC>::T& acc,
                                           const Lanes& L, bool cok, bool own = true) {
  using V = Vec<VEC>;
  const int c0 = L.c0;
  const bool writer = OWN ? own : L.slot == 0;
  const float sc = own ? row_scale(p, row) : 1.f;
  float z[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) {
    const int c = c0 + i;
    z[i] = sc * V::get(acc, i);
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
    const int y = own ? p.labels[row] : -1;
    float zy = 0.f;
#pragma unroll
    for (int i = 0; i < VEC; ++i)
      if (c0 + i == y) zy = z[i];
    zy = group_sum<LANES>(zy);
    if (!writer) return;
    if (L.lane == 0) p.row_loss[row] = (logf(se) + mx) - zy;
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
  } else {
    if constexpr (EPI == AGG_RELU) {
      if (p.relu_bits) {
        // 1[z > 0] of this lane's columns, OR-ed over the lanes of one 32-column word
        // (every lane of the group takes part before any leaves)
        constexpr int kWordLanes = LANES < 32 / VEC ? LANES : 32 / VEC;
        uint32_t bits = 0;
#pragma unroll
        for (int i = 0; i < VEC; ++i)
          if (c0 + i < p.w && z[i] > 0.f) bits |= 1u << ((c0 + i) % 32);
        bits = group_or<kWordLanes>(bits);
        if (writer && c0 < p.w && L.lane % kWordLanes == 0) p.relu_bits[row * p.ld_relu_bits + c0 / 32] = bits;
      }
    }
    if (!cok || !writer) return;
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
      // written once and not read by this kernel: a non-temporal store leaves L2 to the
      // gathered rows
      typedef float f32x4 __attribute__((ext_vector_type(4)));
      const f32x4 o = {z[0], z[VEC > 1 ? 1 : 0], z[VEC > 2 ? 2 : 0], z[VEC > 3 ? 3 : 0]};
      __builtin_nontemporal_store(o, reinterpret_cast<f32x4*>(out));
    } else {
#pragma unroll
      for (int i = 0; i < VEC; ++i)
        if (c0 + i < p.w) out[i] = z[i];
    }
  }
}

// Every row whose length is at most skip_over (all rows when there is no split plan).
// One group per row; the hardware overlaps many resident wavefronts, which hides
// the per-row chain of dependent loads better than prefetching across rows does.
// Group g takes row p.order[g] when the graph carries a row order (long rows first:
// they start early and the short rows fill the end of the launch), else row g.
template <int LANES, int VEC, int EPI>
__global__ void __launch_bounds__(kBlock) k_aggregate(AggParams p, int slots, int64_t skip_over) {
  const Lanes L = lanes_of<LANES, VEC>(slots);
  const bool cok = L.c0 < p.w;
  const int64_t g = (int64_t)blockIdx.x * (kBlock / L.gw) + threadIdx.x / L.gw;
  if constexpr (EPI == AGG_SOFTMAX) {
    // The loss epilogue (row maximum, exponentials, three slice reductions, the loss and
    // the gradient row) would cost every slice of a group the same instructions for one
    // row.  Instead a group sums `slots` consecutive rows one after the other, slice s
    // keeping row s's total, and then every slice finishes its own row.
    const int64_t row0 = g * slots;
    if (row0 >= p.n) return;  // whole groups leave together
    typename Vec<VEC>::T mine = Vec<VEC>::zero();
    bool own = false;
    for (int r = 0; r < slots && row0 + r < p.n; ++r) {
      const int64_t row = p.order ? p.order[row0 + r] : row0 + r;
      const int64_t beg = p.row_ptr[row], end = p.row_ptr[row + 1];
      if (end - beg > skip_over) continue;  // a long row: k_combine finishes it
      const auto acc = accumulate<LANES, VEC>(p, beg, end, L, slots, cok, load_first<LANES>(p, beg, end, L));
      if (L.slot == r) {
        mine = acc;
        own = true;
      }
    }
    const int64_t vr = row0 + L.slot;  // this slice's row, in processing order
    finish_row<LANES, VEC, EPI, true>(p, p.order && vr < p.n ? p.order[vr] : vr, mine, L, cok, own);
  } else {
    if (g >= p.n) return;  // whole groups leave together
    const int64_t row = p.order ? p.order[g] : g;
    const int64_t beg = p.row_ptr[row], end = p.row_ptr[row + 1];
    if (end - beg > skip_over) return;
    const auto acc = accumulate<LANES, VEC>(p, beg, end, L, slots, cok, load_first<LANES>(p, beg, end, L));
    finish_row<LANES, VEC, EPI>(p, row, acc, L, cok);
  }
}

// One group per chunk of a long row: partial[ch, :] = sum over the chunk's entries.
template <int LANES, int VEC>
__global__ void __launch_bounds__(kBlock) k_chunks(AggParams p, gcn_split sp, int slots, float* part, int64_t pw) {
  const Lanes L = lanes_of<LANES, VEC>(slots);
  const int64_t gi = (int64_t)blockIdx.x * (kBlock / L.gw) + threadIdx.x / L.gw;
  if (gi >= sp.n_chunk) return;
  const int64_t ch = sp.order ? sp.order[gi] : gi;
  const int32_t h = sp.owner[ch];
  const int64_t row = sp.rows[h];
  const int64_t beg = p.row_ptr[row] + (ch - sp.first[h]) * (int64_t)GCN_SPLIT_CHUNK;
  const int64_t rend = p.row_ptr[row + 1];
  const int64_t end = beg + GCN_SPLIT_CHUNK < rend ? beg + GCN_SPLIT_CHUNK : rend;
  const bool cok = L.c0 < p.w;
  const auto acc = accumulate<LANES, VEC>(p, beg, end, L, slots, cok, load_first<LANES>(p, beg, end, L));
  if (cok && L.slot == 0) Vec<VEC>::store(part + ch * pw + L.c0, acc);
}

// One group per long row: add its chunk sums in chunk order, then the row epilogue.
template <int LANES, int VEC, int EPI>
__global__ void __launch_bounds__(kBlock) k_combine(AggParams p, gcn_split sp, int slots, const float* part,
                                                    int64_t pw) {
  using V = Vec<VEC>;
  const Lanes L = lanes_of<LANES, VEC>(slots);
  const int64_t h = (int64_t)blockIdx.x * (kBlock / L.gw) + threadIdx.x / L.gw;
  if (h >= sp.n_long) return;
  const bool cok = L.c0 < p.w;
  typename V::T acc = V::zero();
  if (cok)
    for (int64_t ch = sp.first[h]; ch < sp.first[h + 1]; ++ch) V::add(acc, V::load(part + ch * pw + L.c0));
  finish_row<LANES, VEC, EPI>(p, sp.rows[h], acc, L, cok);
}

struct Launch {
  const AggParams* p;
  const gcn_split* sp;
  float* part;
  int64_t pw;
  int slots, chunk_slots;
  hipStream_t s;
};

template <int LANES, int VEC, int EPI>
gcn_status launch3(const Launch& a) {
  const AggParams& p = *a.p;
  const bool split = has_split(a.sp);
  const int64_t skip = split ? (int64_t)GCN_SPLIT_MIN : INT64_MAX;
  const unsigned gy = (unsigned)ceil_div(p.w, LANES * VEC);
  {
    const int gw = LANES * a.slots;
    const int64_t groups = EPI == AGG_SOFTMAX ? ceil_div(p.n, a.slots) : p.n;  // rows per group
    dim3 grid((unsigned)ceil_div(groups, kBlock / gw), gy);
    hipLaunchKernelGGL((k_aggregate<LANES, VEC, EPI>), grid, dim3(kBlock), 0, a.s, p, a.slots, skip);
    GCN_TRY(check_launch("aggregate"));
  }
  if (!split) return GCN_OK;
  {
    const int gw = LANES * a.chunk_slots;
    dim3 grid((unsigned)ceil_div(a.sp->n_chunk, kBlock / gw), gy);
    hipLaunchKernelGGL((k_chunks<LANES, VEC>), grid, dim3(kBlock), 0, a.s, p, *a.sp, a.chunk_slots,
                       a.part, a.pw);
    GCN_TRY(check_launch("aggregate chunks"));
  }
  {
    dim3 grid((unsigned)ceil_div(a.sp->n_long, kBlock / LANES), gy);
    hipLaunchKernelGGL((k_combine<LANES, VEC, EPI>), grid, dim3(kBlock), 0, a.s, p, *a.sp, 1, a.part,
                       a.pw);
    return check_launch("aggregate combine");
  }
}

template <int LANES, int VEC>
gcn_status launch2(const Launch& a) {
  switch (a.p->epi) {
    case AGG_NONE: return launch3<LANES, VEC, AGG_NONE>(a);
    case AGG_RELU: return launch3<LANES, VEC, AGG_RELU>(a);
    case AGG_MASK: return launch3<LANES, VEC, AGG_MASK>(a);
    default: return launch3<LANES, VEC, AGG_SOFTMAX>(a);
  }
}

template <int VEC>
gcn_status launch1(const Launch& a, int lanes) {
  switch (lanes) {
    case 1: return launch2<1, VEC>(a);
    case 2: return launch2<2, VEC>(a);
    case 4: return launch2<4, VEC>(a);
    case 8: return launch2<8, VEC>(a);
    case 16: return launch2<16, VEC>(a);
    case 32: return launch2<32, VEC>(a);
    default: return launch2<64, VEC>(a);
  }
}

// Neighbour slices per row: as many as keep at least one neighbour per slice on an
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
  while (s * 2 <= max_slots && s * 2 <= avg) s *= 2;
  return s;
}

bool use_vec4(const AggParams& p) {
  return p.ldm % 4 == 0 && p.ldz % 4 == 0 && aligned16(p.M) && aligned16(p.Z) &&
         (p.epi != AGG_MASK || (p.ldmask % 4 == 0 && aligned16(p.mask)));
}

}  // namespace

gcn_status launch_aggregate_long_rows(const AggParams& p, const gcn_split* split, void* ws, hipStream_t s) {
  if (!has_split(split) || p.w == 0) return GCN_OK;
  if (!use_vec4(p) || p.epi != AGG_NONE)
    return fail(GCN_E_UNSUPPORTED, "long-row aggregation: needs 16-byte rows and no epilogue");
  int lanes = 1;
  while (lanes < ceil_div(p.w, 4) && lanes < 64) lanes <<= 1;
  const int slots = std::min(64 / lanes, 16);
  const int gw = lanes * slots;
  const unsigned gy = (unsigned)ceil_div(p.w, lanes * 4);
  const int64_t pw = round_up(p.w, 4);
  float* part = static_cast<float*>(ws);
  auto run = [&](auto tag) -> gcn_status {
    constexpr int LN = decltype(tag)::value;
    hipLaunchKernelGGL((k_chunks<LN, 4>), dim3((unsigned)ceil_div(split->n_chunk, kBlock / gw), gy), dim3(kBlock),
                       0, s, p, *split, slots, part, pw);
    GCN_TRY(check_launch("aggregate chunks"));
    hipLaunchKernelGGL((k_combine<LN, 4, AGG_NONE>), dim3((unsigned)ceil_div(split->n_long, kBlock / LN), gy),
                       dim3(kBlock), 0, s, p, *split, 1, part, pw);
    return check_launch("aggregate combine");
  };
  switch (lanes) {
    case 1: return run(std::integral_constant<int, 1>{});
    case 2: return run(std::integral_constant<int, 2>{});
    case 4: return run(std::integral_constant<int, 4>{});
    case 8: return run(std::integral_constant<int, 8>{});
    case 16: return run(std::integral_constant<int, 16>{});
    case 32: return run(std::integral_constant<int, 32>{});
    default: return run(std::integral_constant<int, 64>{});
  }
}

int agg_slots(int lanes, int64_t nnz, int64_t rows) { return pick_slots(lanes, nnz, rows); }

namespace {
// Implicit transpose with atomics (Section IV-D, the CUDA backend's sparse backward):
// C[idx[e], :] += val[e] * B[i, :] for every entry e of compressed row i.  One lane
// group per row reads B's row once and adds it, scaled, into the output row of each
// entry.  Floating-point atomic adds make the order of the additions, and so the
// rounding, vary from run to run.
template <int LANES>
__global__ void __launch_bounds__(256) k_spmm_t_atomic(int64_t nrows, const int64_t* ptr, const int32_t* idx,
                                                       const float* val, const float* B, int64_t ldb, int32_t w,
                                                       float* C, int64_t ldc) {
  const int64_t row = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / LANES;
  const int lane = threadIdx.x % LANES;
  if (row >= nrows) return;
  const int c0 = 4 * lane;
  if (c0 >= w) return;
  const float* b = B + row * ldb + c0;
  float x[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) x[q] = c0 + q < w ? b[q] : 0.f;
  for (int64_t e = ptr[row]; e < ptr[row + 1]; ++e) {
    const float v = val[e];
    float* c = C + (int64_t)idx[e] * ldc + c0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (c0 + q < w) atomicAdd(c + q, v * x[q]);
  }
}

__global__ void __launch_bounds__(256) k_zero_rows(int64_t rows, int32_t w, float* C, int64_t ldc) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < rows * (int64_t)w) C[(i / w) * ldc + i % w] = 0.f;
}

__global__ void k_identity_csr(int32_t n, int64_t* row_ptr, int32_t* col) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i <= n) row_ptr[i] = i;
  if (i < n) col[i] = (int32_t)i;
}
}  // namespace

namespace {
// X^T Q from the CSC view, tiled by row chunks.  Column j of X_csc lists its nonzeros
// (i, x) with i ascending; sum_i x Q[i, :] gathers a row of Q per nonzero, and Q (n rows)
// is far larger than an L2.  Cut the rows into chunks of kXtChunk rows (the chunk's rows
// of Q, at most 8192 x 128 floats = 4 MB, fit one XCD's L2), sum each (column, chunk)
// range into a partial, and give every workgroup of one chunk the same XCD: workgroup
// ids are dealt to the XCDs in turn, so id % 8 names the XCD, and XCD x takes chunks x,
// x + 8, ... one after the other, all columns of a chunk before the next.  The partials
// are added in chunk order afterwards (the same fixed order every run).
constexpr int64_t kXtChunk = 8192;
constexpr int kXcds = 8;

// off[c * F + j] = first entry of column j whose row is >= c * kXtChunk (c = 0..nchunk).
__global__ void __launch_bounds__(256) k_xt_offsets(int32_t F, const int64_t* col_ptr, const int32_t* row,
                                                    int64_t nchunk, int64_t* off) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (nchunk + 1) * F) return;
  const int64_t c = t / F;
  const int32_t j = (int32_t)(t % F);
  int64_t lo = col_ptr[j], hi = col_ptr[j + 1];
  const int64_t r0 = c * kXtChunk;
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (row[mid] < r0) lo = mid + 1;
    else hi = mid;
  }
  off[t] = lo;
}

// part[c][j][0 .. w) = sum over column j's entries in chunk c of x Q[i, :].
template <int LANES, int VEC>
__global__ void __launch_bounds__(kBlock) k_xt_tiled(AggParams p, const int64_t* off, int64_t nchunk,
                                                     int64_t groups, int slots, float* part) {
  const Lanes L = lanes_of<LANES, VEC>(slots);
  const int64_t id = blockIdx.x;
  const int64_t k = id / kXcds;
  const int64_t c = (k / groups) * kXcds + id % kXcds;
  if (c >= nchunk) return;
  const int64_t j = (k % groups) * (kBlock / L.gw) + threadIdx.x / L.gw;
  if (j >= p.n) return;  // whole groups leave together
  const int64_t beg = off[c * p.n + j], end = off[(c + 1) * p.n + j];
  const bool cok = L.c0 < p.w;
  const auto acc = accumulate<LANES, VEC>(p, beg, end, L, slots, cok, load_first<LANES>(p, beg, end, L));
  if (!cok || L.slot != 0) return;
  float* out = part + (c * p.n + j) * p.w + L.c0;
  if (VEC == 4 && p.w % 4 == 0 && L.c0 + 4 <= p.w) {
    Vec<VEC>::store(out, acc);
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i)
      if (L.c0 + i < p.w) out[i] = Vec<VEC>::get(acc, i);
  }
}
}  // namespace

int64_t xt_chunk_rows() { return kXtChunk; }

// GCN_XT=plain keeps the untiled CSC product, =tiled takes the tiled one at any size;
// unset: tiled from four chunks of rows on when a column has at least 16 entries per
// chunk on average.  Measured on the RMAT features (2,097,152 x 4096, w = 128): 1 %
// density 5.87 -> 2.42 ms, 10 % 41.6 -> 19.2 ms, but 0.1 % (about 8 entries per column
// and chunk) 0.62 -> 0.74 ms, where the partials cost more than the gathers save.
bool xt_tiled_enabled(int64_t n, int32_t F, int64_t nnz, int32_t w) {
  if (w <= 0 || w > 256 || F <= 0) return false;
  const char* e = getenv("GCN_XT");
  if (e && strcmp(e, "plain") == 0) return false;
  if (e && strcmp(e, "tiled") == 0) return true;
  const int64_t nchunk = ceil_div(n, kXtChunk);
  return nchunk >= 4 && nnz >= 16 * (int64_t)F * nchunk;
}

size_t xt_tiled_workspace(int64_t n, int32_t F, int32_t w) {
  const int64_t nchunk = std::max<int64_t>(1, ceil_div(n, kXtChunk));
  return (size_t)round_up(8 * (nchunk + 1) * (int64_t)F, 256) + (size_t)round_up(4 * nchunk * (int64_t)F * w, 256);
}

gcn_status launch_spmm_xt_tiled(int64_t n, int32_t F, const int64_t* col_ptr, const int32_t* row, const float* cval,
                                int64_t nnz, const float* B, int64_t ldb, int32_t w, float* C, int64_t ldc, void* ws,
                                hipStream_t s) {
  if (F == 0 || w == 0) return GCN_OK;
  if (w > 256) return fail(GCN_E_UNSUPPORTED, "tiled transpose product: width above 256");
  if (!ws) return fail(GCN_E_INVALID, "tiled transpose product needs a workspace");
  const int64_t nchunk = std::max<int64_t>(1, ceil_div(n, kXtChunk));
  int64_t* off = static_cast<int64_t*>(ws);
  float* part = reinterpret_cast<float*>(static_cast<char*>(ws) + round_up(8 * (nchunk + 1) * (int64_t)F, 256));
  char name[64];
  snprintf(name, sizeof name, "spmm_xtq_tiled_w%d", w);
  ProfScope prof(name, w, F, nnz, s);
  hipLaunchKernelGGL(k_xt_offsets, dim3((unsigned)ceil_div((nchunk + 1) * F, 256)), dim3(256), 0, s, F, col_ptr, row,
                     nchunk, off);
  GCN_TRY(check_launch("tiled transpose offsets"));
  AggParams p{};
  p.n = F;
  p.row_ptr = col_ptr;
  p.col = row;
  p.val = cval;
  p.kind = AGG_W_VAL;
  p.M = B;
  p.ldm = ldb;
  p.w = w;
  const bool vec4 = ldb % 4 == 0 && aligned16(B);
  int lanes = 1;
  while (lanes < ceil_div(w, vec4 ? 4 : 1) && lanes < 64) lanes <<= 1;
  if (!vec4 && w > 64) return fail(GCN_E_UNSUPPORTED, "tiled transpose product: rows of Q must be 16-byte aligned above width 64");
  const int64_t per_col = std::max<int64_t>(1, nnz / std::max<int64_t>(1, (int64_t)F * nchunk));
  const int slots = pick_slots(lanes, per_col * F, F);
  const int gw = lanes * slots;
  const int64_t groups = ceil_div(F, kBlock / gw);
  const int64_t grid = ceil_div(nchunk, kXcds) * kXcds * groups;
  if (grid > INT32_MAX) return fail(GCN_E_RANGE, "tiled transpose product: too many workgroups");
  auto run = [&](auto ln, auto vc) {
    constexpr int LN = decltype(ln)::value, VC = decltype(vc)::value;
    hipLaunchKernelGGL((k_xt_tiled<LN, VC>), dim3((unsigned)grid), dim3(kBlock), 0, s, p, off, nchunk, groups, slots,
                       part);
  };
  using I = std::integral_constant<int, 4>;
  using O = std::integral_constant<int, 1>;
  switch (lanes) {
    case 1: vec4 ? run(std::integral_constant<int, 1>{}, I{}) : run(std::integral_constant<int, 1>{}, O{}); break;
    case 2: vec4 ? run(std::integral_constant<int, 2>{}, I{}) : run(std::integral_constant<int, 2>{}, O{}); break;
    case 4: vec4 ? run(std::integral_constant<int, 4>{}, I{}) : run(std::integral_constant<int, 4>{}, O{}); break;
    case 8: vec4 ? run(std::integral_constant<int, 8>{}, I{}) : run(std::integral_constant<int, 8>{}, O{}); break;
    case 16: vec4 ? run(std::integral_constant<int, 16>{}, I{}) : run(std::integral_constant<int, 16>{}, O{}); break;
    case 32: vec4 ? run(std::integral_constant<int, 32>{}, I{}) : run(std::integral_constant<int, 32>{}, O{}); break;
    default: vec4 ? run(std::integral_constant<int, 64>{}, I{}) : run(std::integral_constant<int, 64>{}, O{}); break;
  }
  GCN_TRY(check_launch("tiled transpose product"));
  return launch_partial_sum(part, nchunk, F, w, C, ldc, s);
}

size_t spmm_xt_workspace(int64_t n, int32_t F, int64_t nnz, int32_t w, const gcn_split* csc_split) {
  if (xt_tiled_enabled(n, F, nnz, w)) return xt_tiled_workspace(n, F, w);
  return aggregate_workspace(csc_split, w);
}

gcn_status launch_spmm_xt(int64_t n, int32_t F, int64_t nnz, const int64_t* col_ptr, const int32_t* row,
                          const float* cval, const gcn_split* csc_split, const float* B, int64_t ldb, int32_t w,
                          float* C, int64_t ldc, void* ws, hipStream_t s) {
  if (xt_tiled_enabled(n, F, nnz, w))
    return launch_spmm_xt_tiled(n, F, col_ptr, row, cval, nnz, B, ldb, w, C, ldc, ws, s);
  AggParams p{};
  p.n = F;
  p.row_ptr = col_ptr;
  p.col = row;
  p.val = cval;
  p.M = B;
  p.ldm = ldb;
  p.w = w;
  p.Z = C;
  p.ldz = ldc;
  p.epi = AGG_NONE;
  p.tag = "spmm_xtq";
  return launch_aggregate(p, nnz, csc_split, ws, s);
}

gcn_status launch_spmm_t_atomic(int64_t nrows, const int64_t* ptr, const int32_t* idx, const float* val,
                                const float* B, int64_t ldb, int32_t w, int64_t out_rows, float* C, int64_t ldc,
                                int64_t nnz, hipStream_t s) {
  if (out_rows > 0 && w > 0) {
    hipLaunchKernelGGL(k_zero_rows, dim3((unsigned)ceil_div(out_rows * w, 256)), dim3(256), 0, s, out_rows, w, C,
                       ldc);
    GCN_TRY(check_launch("zero rows"));
  }
  if (nrows == 0 || w == 0) return GCN_OK;
  char name[64];
  snprintf(name, sizeof name, "spmm_t_atomic_w%d", w);
  ProfScope prof(name, w, nrows, nnz, s);
  if (w <= 64) {
    hipLaunchKernelGGL(k_spmm_t_atomic<16>, dim3((unsigned)ceil_div(nrows * 16, 256)), dim3(256), 0, s, nrows,
                       ptr, idx, val, B, ldb, w, C, ldc);
  } else if (w <= 128) {
    hipLaunchKernelGGL(k_spmm_t_atomic<32>, dim3((unsigned)ceil_div(nrows * 32, 256)), dim3(256), 0, s, nrows,
                       ptr, idx, val, B, ldb, w, C, ldc);
  } else if (w <= 256) {
    hipLaunchKernelGGL(k_spmm_t_atomic<64>, dim3((unsigned)ceil_div(nrows * 64, 256)), dim3(256), 0, s, nrows,
                       ptr, idx, val, B, ldb, w, C, ldc);
  } else {
    return fail(GCN_E_UNSUPPORTED, "atomic transpose product: width above 256");
  }
  return check_launch("atomic transpose product");
}

gcn_status launch_identity_csr(int32_t n, int64_t* row_ptr, int32_t* col, hipStream_t s) {
  hipLaunchKernelGGL(k_identity_csr, dim3((unsigned)ceil_div((int64_t)n + 1, 256)), dim3(256), 0, s, n, row_ptr,
                     col);
  return check_launch("identity operator");
}

size_t aggregate_workspace(const gcn_split* split, int32_t w) {
  if (!has_split(split)) return 0;
  return sizeof(float) * (size_t)split->n_chunk * (size_t)round_up(w, 4);
}

gcn_status launch_aggregate(const AggParams& p, int64_t nnz, const gcn_split* split, void* ws,
                            hipStream_t s) {
  if (p.n == 0 || p.w == 0) return GCN_OK;
  const bool vec4 = use_vec4(p);
  const int vec = vec4 ? 4 : 1;
  int need = (int)ceil_div(p.w, vec);
  // A slice spans at most 32 lanes (128 columns with 16-byte loads); wider rows take
  // several column groups (blockIdx.y), which are dispatched one after the other, so a
  // 256-wide aggregation gathers 512-byte half rows in two passes.  The 32-lane kernel
  // holds 71 VGPRs (7 wavefronts per SIMD) against 112 (4) for a 64-lane slice, and runs
  // 256-wide rows about 10 % faster.  The softmax epilogue needs the whole row in one
  // slice, so it keeps up to 64 lanes.
  const int max_lanes = p.epi == AGG_SOFTMAX ? 64 : 32;
  int lanes = 1;
  while (lanes < need && lanes < max_lanes) lanes <<= 1;
  if (p.epi == AGG_SOFTMAX && need > lanes)
    return fail(GCN_E_UNSUPPORTED, "softmax epilogue needs width <= 256 (vector) or 64 (scalar)");
  if (has_split(split) && !ws) return fail(GCN_E_INVALID, "aggregation of split rows needs a workspace");
  // The row order costs every row a scattered read of its offsets and a scattered write of
  // its output row; it pays where a row gathers enough bytes to hide that: taken from 4 KB
  // of gathered rows per average row on (measured on arxiv-like, 14.7 entries per row:
  // width 40 +18 % with the order, widths 128 and 256 -23 % and -10 %).
  AggParams q = p;
  if (q.order && nnz >= 0 && (double)nnz / (double)p.n * 4.0 * (double)p.w < 4096.0) q.order = nullptr;
  Launch a;
  a.p = &q;
  a.sp = split;
  a.part = static_cast<float*>(ws);
  a.pw = round_up(p.w, 4);
  a.slots = pick_slots(lanes, nnz, p.n);
  a.chunk_slots = std::min(64 / lanes, 16);
  a.s = s;
  char name[64];
  snprintf(name, sizeof name, "%s_w%d", p.tag ? p.tag : "aggregate", p.w);
  ProfScope prof(name, p.w, p.n, nnz, s);
  return vec4 ? launch1<4>(a, lanes) : launch1<1>(a, lanes);
}

}  // namespace gcn
