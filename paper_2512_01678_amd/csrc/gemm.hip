// gemm.hip -- dense fp32 products on the gfx950 matrix cores.
//
// The dense-path transforms of Algorithm 1 (GEMM(X, W) forward, GEMM^T(X, G)
// backward) plus the input-gradient product Q W^T of backpropagation:
//   C(m, n) = sum_k A(m, k) B(k, n)
// with either operand read transposed.  One workgroup computes a BM x BN tile
// with WM x WN wavefronts, each issuing v_mfma_f32_32x32x2_f32 on 32 x 32
// sub-tiles.  K is walked in BK-wide slabs staged through LDS with two
// buffers: the next slab's global loads are in flight while the matrix cores
// work on the current one.  Each operand is staged in the layout it has in
// memory (no transposing stores): "k-contiguous" slabs are read back as
// 16-byte vectors, "m/n-contiguous" slabs as one conflict-free dword per lane.
// The k index inside a slab is permuted consistently for A and B (lane half h
// takes k = h*BK/2 + kk), which a sum over k does not notice.
//
// Epilogues: + bias, ReLU, or multiplication by 1[mask > 0]; or, for a
// split-k launch, a plain store of the partial tile into the workspace, summed
// afterwards in a fixed order by k_splitk_reduce (deterministic, no atomics).
//
// Two arithmetic modes give fp32 results:
//  * fp32: v_mfma_f32_32x32x2_f32 on the fp32 operands;
//  * bf16x6 (default): every fp32 operand is split exactly into three bf16 parts
//    a = a_hi + a_mid + a_lo (24 significant bits, each subtraction exact in
//    fp32), and the six cross products of order <= 2 (hi.hi, hi.mid, mid.hi,
//    hi.lo, mid.mid, lo.hi) run on v_mfma_f32_32x32x16_bf16 with fp32
//    accumulation; bf16 x bf16 products are exact in fp32 and the dropped terms
//    are below 2^-24 of |a b|, so the result carries fp32 accuracy at 6 bf16
//    instructions per 32x32x16 step instead of 8 fp32 ones at a quarter of the
//    rate.  The split happens once per element, when a slab is staged: LDS holds
//    three k-contiguous bf16 planes, so the wavefronts that share an operand row
//    do not each redo it (vector ALU time, not the matrix cores, bounds this
//    product on gfx950), and every fragment is one 16-byte LDS read.
#include <cstring>

#include "bf16x6.h"

namespace gcn {
namespace {


constexpr int kPad = 4;
typedef float f32x4 __attribute__((ext_vector_type(4)));


struct GemmArgs {
  GemmParams p;
  float* part;     // split-k partial tiles (split index major), or NULL
  int64_t kchunk;  // k extent per split
  int a_vec;       // A rows are 16-byte aligned with pitch % 4 == 0
  int b_vec;
  int o_vec;       // output rows (C, or the split-k partials) likewise
  int m_vec;       // mask rows likewise
};

// Load 4 consecutive elements src[i .. i+3] (i < lim are valid) into v.
__device__ __forceinline__ float4 load4(const float* src, int64_t i, int64_t lim, bool vec) {
  if (vec && i + 4 <= lim) return *reinterpret_cast<const float4*>(src + i);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (i + 0 < lim) v.x = src[i + 0];
  if (i + 1 < lim) v.y = src[i + 1];
  if (i + 2 < lim) v.z = src[i + 2];
  if (i + 3 < lim) v.w = src[i + 3];
  return v;
}

// Staging of one operand slab.  Operand X(r, k) with r in [r0, r0+R) (r < rlim)
// and k in [k0, k0+BK) (k < klim).  KCONT: X(r,k) = src[r*ld + k], else
// src[k*ld + r].  LDS layout: KCONT -> [R][BK+kPad], else [BK][R+kPad].
template <int R, int BK, int NT, bool KCONT>
struct Stage {
  static constexpr int kChunks = R * BK / 4;
  static constexpr int kPer = (kChunks + NT - 1) / NT;
  static constexpr int kLdsFloats = KCONT ? R * (BK + kPad) : BK * (R + kPad);
  float4 reg[kPer];
  const float* src_;
  int64_t ld_, r0_, rlim_, kend_;
  bool vec_;

  __device__ __forceinline__ void prepare(const float* src, int64_t ld, int64_t r0, int64_t rlim,
                                          int64_t kend, bool vec, int) {
    src_ = src;
    ld_ = ld;
    r0_ = r0;
    rlim_ = rlim;
    kend_ = kend;
    vec_ = vec;
  }
  __device__ __forceinline__ void load(int64_t k0, int tid) { load(src_, ld_, r0_, rlim_, k0, kend_, vec_, tid); }
  __device__ __forceinline__ void load(const float* src, int64_t ld, int64_t r0, int64_t rlim,
                                       int64_t k0, int64_t klim, bool vec, int tid) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = tid + i * NT;
      reg[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (c < kChunks) {
        if (KCONT) {
          const int r = c / (BK / 4), kq = (c % (BK / 4)) * 4;
          if (r0 + r < rlim) reg[i] = load4(src + (r0 + r) * ld, k0 + kq, klim, vec);
        } else {
          const int kr = c / (R / 4), rq = (c % (R / 4)) * 4;
          if (k0 + kr < klim) reg[i] = load4(src + (k0 + kr) * ld, r0 + rq, rlim, vec);
        }
      }
    }
  }
  __device__ __forceinline__ void store(float* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = tid + i * NT;
      if (c < kChunks) {
        if (KCONT) {
          const int r = c / (BK / 4), kq = (c % (BK / 4)) * 4;
          *reinterpret_cast<float4*>(lds + r * (BK + kPad) + kq) = reg[i];
        } else {
          const int kr = c / (R / 4), rq = (c % (R / 4)) * 4;
          *reinterpret_cast<float4*>(lds + kr * (R + kPad) + rq) = reg[i];
        }
      }
    }
  }
  // fragment value for sub-tile row rr (0..R-1), slab k index kidx
  static __device__ __forceinline__ float frag(const float* lds, int rr, int kidx) {
    return KCONT ? lds[rr * (BK + kPad) + kidx] : lds[kidx * (R + kPad) + rr];
  }
};

// Staging of one operand slab for the bf16x6 mode: every element is split once, when
// the slab goes into LDS, into three bf16 planes laid out k-contiguous,
// [plane][R][BK + 8], so that a fragment (8 consecutive k of one row) is one 16-byte
// read.  Each thread loads 4 consecutive k of one row: a 16-byte vector when k is
// contiguous in memory, else 4 dwords that are coalesced across the lanes (consecutive
// lanes take consecutive rows).  A thread's byte offsets inside the tile are fixed for
// the whole k walk, so a slab load is a wave-uniform base plus those 32-bit offsets
// (no per-slab address arithmetic); rows past the edge of the matrix re-read its last
// row (their outputs are never stored); only a partial last slab checks k.
template <int R, int BK, int NT, bool KCONT>
struct StageX {
  static constexpr int kChunks = R * BK / 4;
  static constexpr int kPer = (kChunks + NT - 1) / NT;
  static constexpr int kPitch = BK + 8;  // bf16 per plane row (16-byte multiple)
  static constexpr int kPlane = R * kPitch;
  static constexpr int kLdsFloats = 3 * kPlane / 2;
  float4 reg[kPer];
  uint32_t off[kPer];  // byte offset of the chunk's first element from the slab base
  const char* src;
  int64_t ld, r0, kend;
  bool vec;

  static __device__ __forceinline__ void coords(int c, int& r, int& kq) {
    if (KCONT) {
      r = c / (BK / 4);
      kq = (c % (BK / 4)) * 4;
    } else {
      r = c % R;
      kq = (c / R) * 4;
    }
  }
  __device__ __forceinline__ void prepare(const float* src_, int64_t ld_, int64_t r0_, int64_t rlim,
                                          int64_t kend_, bool vec_, int tid) {
    src = reinterpret_cast<const char*>(src_);
    ld = ld_;
    r0 = r0_;
    kend = kend_;
    vec = vec_;
    const int64_t last = rlim - 1 - r0_;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      int r, kq;
      coords(tid + i * NT, r, kq);
      const int64_t rr = r < last ? r : last;
      off[i] = (uint32_t)(4 * (KCONT ? rr * ld + kq : kq * ld + rr));
    }
  }
  __device__ __forceinline__ void load(int64_t k0, int tid) {
    const char* base = src + 4 * (KCONT ? r0 * ld + k0 : k0 * ld + r0);
    const int64_t kleft = kend - k0;  // >= 1
    if (kleft >= BK && (vec || !KCONT)) {
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        if (kChunks % NT == 0 || tid + i * NT < kChunks) {
          if (KCONT) {
            reg[i] = *reinterpret_cast<const float4*>(base + off[i]);
          } else {
            const char* q = base + off[i];
            reg[i].x = *reinterpret_cast<const float*>(q);
            reg[i].y = *reinterpret_cast<const float*>(q + 4 * ld);
            reg[i].z = *reinterpret_cast<const float*>(q + 8 * ld);
            reg[i].w = *reinterpret_cast<const float*>(q + 12 * ld);
          }
        }
      }
    } else {
      // partial last slab, or unaligned k-contiguous rows: element by element
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        reg[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        int r, kq;
        coords(tid + i * NT, r, kq);
        if (kChunks % NT == 0 || tid + i * NT < kChunks) {
          const char* q = base + off[i];
          const int64_t step = KCONT ? 4 : 4 * ld;
          if (kq + 0 < kleft) reg[i].x = *reinterpret_cast<const float*>(q);
          if (kq + 1 < kleft) reg[i].y = *reinterpret_cast<const float*>(q + step);
          if (kq + 2 < kleft) reg[i].z = *reinterpret_cast<const float*>(q + 2 * step);
          if (kq + 3 < kleft) reg[i].w = *reinterpret_cast<const float*>(q + 3 * step);
        }
      }
    }
  }
  __device__ __forceinline__ void store(float* lds_f, int tid) const {
    __bf16* lds = reinterpret_cast<__bf16*>(lds_f);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int c = tid + i * NT;
      if (kChunks % NT == 0 || c < kChunks) {
        int r, kq;
        coords(c, r, kq);
        uint2 hi, mid, lo;
        split_pair(reg[i].x, reg[i].y, hi.x, mid.x, lo.x);
        split_pair(reg[i].z, reg[i].w, hi.y, mid.y, lo.y);
        __bf16* d = lds + r * kPitch + kq;
        *reinterpret_cast<uint2*>(d) = hi;
        *reinterpret_cast<uint2*>(d + kPlane) = mid;
        *reinterpret_cast<uint2*>(d + 2 * kPlane) = lo;
      }
    }
  }
  // 8 consecutive k (from kofs) of sub-tile row rr in plane pl
  static __device__ __forceinline__ bf16x8 frag(const float* lds_f, int pl, int rr, int kofs) {
    const __bf16* lds = reinterpret_cast<const __bf16*>(lds_f);
    return *reinterpret_cast<const bf16x8*>(lds + pl * kPlane + rr * kPitch + kofs);
  }
};

template <bool EMU, int R, int BK, int NT, bool KCONT>
struct StageFor {
  using T = Stage<R, BK, NT, KCONT>;
};
template <int R, int BK, int NT, bool KCONT>
struct StageFor<true, R, BK, NT, KCONT> {
  using T = StageX<R, BK, NT, KCONT>;
};

template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB, int EPI, bool SPLIT, bool EMU>
__global__ void __launch_bounds__(WM* WN * 64) k_gemm(GemmArgs g) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / WM / 32;
  constexpr int TN = BN / WN / 32;
  constexpr int KH = BK / 2;
  using SA = typename StageFor<EMU, BM, BK, NT, !TA>::T;  // A(m,k): k-contiguous unless transposed
  using SB = typename StageFor<EMU, BN, BK, NT, TB>::T;   // B(k,n): n-contiguous unless transposed
  // LDS buffers per operand: two for fp32 slabs (the next slab is stored while the
  // current one is read); one for the larger bf16 planes (the next slab waits in
  // registers behind an extra barrier), which leaves room for more workgroups per CU
  constexpr int NBUF = EMU ? 1 : 2;
  constexpr int kA = SA::kLdsFloats, kB = SB::kLdsFloats;
  constexpr int RB = BM / WM;               // rows of one epilogue round
  constexpr int kEpi = RB * (BN + kPad);
  constexpr int kTot = NBUF * (kA + kB) > kEpi ? NBUF * (kA + kB) : kEpi;
  __shared__ __attribute__((aligned(16))) float smem[kTot];
  auto lds_a = [&](int b) { return smem + (b % NBUF) * kA; };
  auto lds_b = [&](int b) { return smem + NBUF * kA + (b % NBUF) * kB; };

  const GemmParams& p = g.p;
  const int tid = threadIdx.x;
  const int wave = tid / 64, l = tid % 64;
  const int wm = wave % WM, wn = wave / WM;
  const int h = l / 32, l32 = l % 32;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int64_t n0 = (int64_t)blockIdx.y * BN;
  int64_t kbeg = 0, kend = p.k;
  if (SPLIT) {
    kbeg = (int64_t)blockIdx.z * g.kchunk;
    kend = kbeg + g.kchunk < p.k ? kbeg + g.kchunk : p.k;
  }

  floatx16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  SA sa;
  SB sb;
  // A operand: rows m, cols k.  TA: stored k x m.
  sa.prepare(p.A, p.lda, m0, p.m, kend, g.a_vec, tid);
  sb.prepare(p.B, p.ldb, n0, p.n, kend, g.b_vec, tid);
  auto load_slab = [&](int64_t k0) {
    sa.load(k0, tid);
    sb.load(k0, tid);
  };

  const int64_t nslab = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  if (nslab > 0) {
    load_slab(kbeg);
    sa.store(lds_a(0), tid);
    sb.store(lds_b(0), tid);
  }
  __syncthreads();
  for (int64_t s = 0; s < nslab; ++s) {
    const int buf = (int)(s & 1);
    if (s + 1 < nslab) load_slab(kbeg + (s + 1) * BK);
    const float* la = lds_a(buf);
    const float* lb = lds_b(buf);
    if constexpr (EMU) {
      // BK / 16 steps of 32x32x16 per slab; in step t lane half h holds
      // k = h * BK / 2 + 8 t .. + 7 of both operands
#pragma unroll
      for (int t = 0; t < BK / 16; ++t) {
        bf16x8 ah[TM], am[TM], al[TM], bh[TN], bm[TN], bl[TN];
        const int kofs = h * KH + 8 * t;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int rr = wm * (BM / WM) + i * 32 + l32;
          ah[i] = SA::frag(la, 0, rr, kofs);
          am[i] = SA::frag(la, 1, rr, kofs);
          al[i] = SA::frag(la, 2, rr, kofs);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int rr = wn * (BN / WN) + j * 32 + l32;
          bh[j] = SB::frag(lb, 0, rr, kofs);
          bm[j] = SB::frag(lb, 1, rr, kofs);
          bl[j] = SB::frag(lb, 2, rr, kofs);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[i], bh[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am[i], bm[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[i], bl[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am[i], bh[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[i], bm[j], acc[i][j], 0, 0, 0);
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[i], bh[j], acc[i][j], 0, 0, 0);
          }
      }
    } else {
      float af[TM][KH], bf[TN][KH];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int kk = 0; kk < KH; ++kk) af[i][kk] = SA::frag(la, wm * (BM / WM) + i * 32 + l32, h * KH + kk);
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int kk = 0; kk < KH; ++kk) bf[j][kk] = SB::frag(lb, wn * (BN / WN) + j * 32 + l32, h * KH + kk);
#pragma unroll
      for (int kk = 0; kk < KH; ++kk)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[i][kk], bf[j][kk], acc[i][j], 0, 0, 0);
    }
    if (NBUF == 1) __syncthreads();  // every wave is done with the only buffer
    if (s + 1 < nslab) {
      sa.store(lds_a(buf ^ 1), tid);
      sb.store(lds_b(buf ^ 1), tid);
    }
    __syncthreads();
  }

  // Epilogue, one wave-row of the tile (RB rows) per round: the waves of that row
  // put their accumulators in LDS (lane l32 holds column l32 of a 32x32 sub-tile,
  // register r row 8*(r/4) + 4*h + r%4), then the whole workgroup streams the RB x BN
  // slab out as row-contiguous 16-byte accesses (mask, bias, C or the split-k partial);
  // the mask and C streams are touched once (non-temporal, leaving L2 to the operands).
  // Split-k partials are stored normally: the reduce reads them back at once.
  float* const tile = smem;
  const int64_t ldo = SPLIT ? p.n : p.ldc;
  float* const out = SPLIT ? g.part + (int64_t)blockIdx.z * p.m * p.n : p.C;
  const bool ovec = g.o_vec;
  const bool mvec = g.m_vec;
  for (int round = 0; round < WM; ++round) {
    if (wm == round) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            tile[(i * 32 + 8 * (r / 4) + 4 * h + (r % 4)) * (BN + kPad) + wn * (BN / WN) + j * 32 + l32] =
                acc[i][j][r];
    }
    __syncthreads();
    constexpr int kChunks = RB * BN / 4;
    for (int c = tid; c < kChunks; c += NT) {
      const int rr = c / (BN / 4), cq = (c % (BN / 4)) * 4;
      const int64_t row = m0 + (int64_t)round * RB + rr;
      const int64_t col = n0 + cq;
      if (row >= p.m || col >= p.n) continue;
      float v[4];
      const float4 t4 = *reinterpret_cast<const float4*>(tile + rr * (BN + kPad) + cq);
      v[0] = t4.x; v[1] = t4.y; v[2] = t4.z; v[3] = t4.w;
      const bool full = col + 4 <= p.n;
      if (!SPLIT) {
        float mk[4] = {1.f, 1.f, 1.f, 1.f};
        if (EPI == GEMM_MASK) {
          const float* mp = p.mask + row * p.ldmask + col;
          if (mvec && full) {
            const f32x4 m4 = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(mp));
            mk[0] = m4[0]; mk[1] = m4[1]; mk[2] = m4[2]; mk[3] = m4[3];
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) mk[q] = col + q < p.n ? mp[q] : 0.f;
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (p.bias && col + q < p.n) v[q] += p.bias[col + q];
          if (EPI == GEMM_RELU) v[q] = fmaxf(v[q], 0.f);
          if (EPI == GEMM_MASK) v[q] = mk[q] > 0.f ? v[q] : 0.f;
        }
      }
      float* op = out + row * ldo + col;
      if (ovec && full) {
        const f32x4 o = {v[0], v[1], v[2], v[3]};
        if (SPLIT) *reinterpret_cast<f32x4*>(op) = o;  // partials: read back at once by the reduce
        else __builtin_nontemporal_store(o, reinterpret_cast<f32x4*>(op));
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (col + q < p.n) op[q] = v[q];
      }
    }
    __syncthreads();
  }
}

// C(m,n) = sum_s part[s](m,n) (+ bias).  A workgroup owns kRedElems = 256 / SL
// consecutive output elements; its SL split lanes sum the partials s = lane, lane + SL,
// ... in increasing order into four interleaved accumulators, and the SL lane sums are
// combined by a fixed binary tree, so the rounding is fixed.  SL = 4 reads 256-byte
// segments of each partial; SL = 16 (64-byte segments) keeps each lane's chain of
// dependent loads short when the output is small and the splits are many (the 256 x 40
// weight gradient sums 512 partials).
template <int SL>
__global__ void __launch_bounds__(256) k_splitk_reduce(const float* part, int64_t splits, int64_t m,
                                                       int64_t n, float* C, int64_t ldc,
                                                       const float* bias) {
  constexpr int kRedLanes = SL, kRedElems = 256 / SL;
  __shared__ float red[kRedLanes][kRedElems];
  const int e = threadIdx.x % kRedElems, sl = threadIdx.x / kRedElems;
  const int64_t i = (int64_t)blockIdx.x * kRedElems + e;
  const int64_t mn = m * n;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  if (i < mn) {
    int64_t z = sl;
    for (; z + 3 * kRedLanes < splits; z += 4 * kRedLanes) {
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] += part[(z + kRedLanes * u) * mn + i];
    }
    for (; z < splits; z += kRedLanes) acc[0] += part[z * mn + i];
  }
  red[sl][e] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  __syncthreads();
  for (int o = kRedLanes / 2; o > 0; o >>= 1) {
    if (sl < o) red[sl][e] += red[sl + o][e];
    __syncthreads();
  }
  if (sl == 0 && i < mn) {
    float s = red[0][e];
    const int64_t row = i / n, col = i % n;
    if (bias) s += bias[col];
    C[row * ldc + col] = s;
  }
}

// Launch of k_splitk_reduce: 16 split lanes when the 4-lane form would leave the CUs with
// fewer than two workgroups each.
gcn_status launch_reduce(const float* part, int64_t splits, int64_t m, int64_t n, float* C, int64_t ldc,
                         const float* bias, hipStream_t s) {
  const int64_t total = m * n;
  if (ceil_div(total, 64) < 512)
    hipLaunchKernelGGL(k_splitk_reduce<16>, dim3((unsigned)ceil_div(total, 16)), dim3(256), 0, s, part, splits, m, n,
                       C, ldc, bias);
  else
    hipLaunchKernelGGL(k_splitk_reduce<4>, dim3((unsigned)ceil_div(total, 64)), dim3(256), 0, s, part, splits, m, n,
                       C, ldc, bias);
  return check_launch("split-k reduce");
}

}  // namespace

gcn_status launch_partial_sum(const float* part, int64_t splits, int64_t m, int64_t n, float* C, int64_t ldc,
                              hipStream_t s) {
  const int64_t total = m * n;
  if (total == 0) return GCN_OK;
  return launch_reduce(part, splits, m, n, C, ldc, nullptr, s);
}

namespace {
struct Shape {
  int bm, bn;
};

// 128 x 128 tiles (2 x 2 wavefronts) for wide outputs; for narrow ones BM x 32 or BM x 64
// tiles of BM / 64 wavefronts stacked along m: 256 rows in fp32 mode, 128 in bf16x6 mode
// (whose larger LDS slabs would otherwise hold a CU to one workgroup).
Shape pick_shape(const GemmParams& p, bool emu) {
  const int bm = emu ? 128 : 256;
  if (p.n <= 32) return {bm, 32};
  if (p.n <= 64) return {bm, 64};
  // A^T B (weight gradients, split k) with both sides above 128: one 256 x 256 tile
  // (8 wavefronts) reads each operand once instead of twice (arxiv-like 256 x 256:
  // 142 -> 126 us; a 128 x 256 tile for the 128-wide case was slower than 128 x 128)
  if (p.ta && emu && p.n > 128 && p.m > 128) return {256, 256};
  return {128, 128};
}

#ifndef GCN_TN_WAVES
#define GCN_TN_WAVES 2048  // wavefronts of a split-k A^T B launch
#endif

int64_t pick_splits(const GemmParams& p, Shape sh) {
  if (!p.ta) return 1;  // only A^T B reduces over the long (row) dimension
  // about 2048 wavefronts in all (measured best for wide and narrow tiles alike), each
  // workgroup walking at least 256 rows of k
  const int64_t tiles = ceil_div(p.m, sh.bm) * ceil_div(p.n, sh.bn);
  const int64_t waves = sh.bn >= 256 ? 8 : (sh.bn >= 128 ? 4 : sh.bm / 64);
  int64_t s = ceil_div(GCN_TN_WAVES, tiles * waves);
  const int64_t max_s = ceil_div(p.k, 256);
  if (s > max_s) s = max_s;
  return s < 1 ? 1 : s;
}

template <int BM, int BN, int BK, int WM, int WN, bool TA, bool TB, bool EMU>
gcn_status launch_tile(const GemmArgs& g, int64_t splits, hipStream_t s) {
  dim3 grid((unsigned)ceil_div(g.p.m, BM), (unsigned)ceil_div(g.p.n, BN), (unsigned)splits);
  dim3 block(WM * WN * 64);
  if (splits > 1) {
    hipLaunchKernelGGL((k_gemm<BM, BN, BK, WM, WN, TA, TB, GEMM_NONE, true, EMU>), grid, block, 0, s, g);
  } else {
    switch (g.p.epi) {
      case GEMM_RELU:
        hipLaunchKernelGGL((k_gemm<BM, BN, BK, WM, WN, TA, TB, GEMM_RELU, false, EMU>), grid, block, 0, s, g);
        break;
      case GEMM_MASK:
        hipLaunchKernelGGL((k_gemm<BM, BN, BK, WM, WN, TA, TB, GEMM_MASK, false, EMU>), grid, block, 0, s, g);
        break;
      default:
        hipLaunchKernelGGL((k_gemm<BM, BN, BK, WM, WN, TA, TB, GEMM_NONE, false, EMU>), grid, block, 0, s, g);
    }
  }
  return check_launch("gemm");
}

// Slab depth: 16, except 32 for the plain (NN) bf16x6 product on wide tiles, whose
// operands both stream from contiguous rows (measured fastest per layout).
template <bool TA, bool TB, bool EMU>
gcn_status launch_shape(const GemmArgs& g, Shape sh, int64_t splits, hipStream_t s) {
  constexpr int BKW = (EMU && !TA && !TB) ? 32 : 16;
  constexpr int BMN = EMU ? 128 : 256, WMN = BMN / 64;
  if (sh.bn == 32) return launch_tile<BMN, 32, 16, WMN, 1, TA, TB, EMU>(g, splits, s);
  if (sh.bn == 64) return launch_tile<BMN, 64, 16, WMN, 1, TA, TB, EMU>(g, splits, s);
  if constexpr (TA && !TB && EMU) {
    if (sh.bn == 256) return launch_tile<256, 256, 16, 2, 4, TA, TB, EMU>(g, splits, s);
  }
  return launch_tile<128, 128, BKW, 2, 2, TA, TB, EMU>(g, splits, s);
}

template <bool TA, bool TB>
gcn_status launch_layout(const GemmArgs& g, Shape sh, int64_t splits, bool emu, hipStream_t s) {
  return emu ? launch_shape<TA, TB, true>(g, sh, splits, s) : launch_shape<TA, TB, false>(g, sh, splits, s);
}

// Arithmetic mode: bf16x6 unless GCN_GEMM_MODE=fp32 (native fp32 MFMA, kept for comparison).
// The bf16x6 staging addresses a tile with 32-bit offsets (R * ld * 4 bytes for a
// k-contiguous operand, R <= 256 rows; 16 * ld * 4 for the other layout); operands with
// larger pitches take the fp32 mode.
bool use_emulation(const GemmParams& p) {
  if (!gemm_bf16x6_mode()) return false;
  const int64_t lim = (int64_t)1 << 31;
  return (p.ta ? 16 * p.lda : 256 * p.lda) * 4 < lim && (p.tb ? 256 * p.ldb : 16 * p.ldb) * 4 < lim;
}

}  // namespace

bool gemm_bf16x6_mode() {
  const char* e = getenv("GCN_GEMM_MODE");
  return !(e && strcmp(e, "fp32") == 0);
}

bool gemm_split_k(const GemmParams& p) {
  return !gemm_rows_supported(p) && p.k > 0 && pick_splits(p, pick_shape(p, use_emulation(p))) > 1;
}

size_t gemm_workspace(const GemmParams& p) {
  if (gemm_rows_supported(p)) return gemm_rows_workspace(p);
  const Shape sh = pick_shape(p, use_emulation(p));
  const int64_t s = pick_splits(p, sh);
  return s > 1 ? sizeof(float) * (size_t)(s * p.m * p.n) : 0;
}

gcn_status launch_gemm(const GemmParams& p, void* ws, hipStream_t s) {
  if (p.m == 0 || p.n == 0) return GCN_OK;
  if ((p.mask_bits || p.relu_bits) && !gemm_rows_supported(p))
    return fail(GCN_E_UNSUPPORTED, "gemm: bitmask epilogues need the row-panel product");
  if (gemm_rows_supported(p)) {
    if (!ws) return fail(GCN_E_INVALID, "gemm: the row-panel product needs its workspace");
    char name[64];
    snprintf(name, sizeof name, "gemm_%s_%ldx%ldx%ld", p.tb ? "NT" : "NN", (long)p.m, (long)p.n, (long)p.k);
    ProfScope prof(name, (int32_t)p.n, p.m, p.k, s);
    return launch_gemm_rows(p, ws, s);
  }
  const bool emu = use_emulation(p);
  const Shape sh = pick_shape(p, emu);
  const int64_t splits = p.k == 0 ? 1 : pick_splits(p, sh);
  GemmArgs g;
  g.p = p;
  g.part = splits > 1 ? static_cast<float*>(ws) : nullptr;
  g.kchunk = round_up(ceil_div(p.k, splits), 16);
  g.a_vec = p.lda % 4 == 0 && aligned16(p.A);
  g.b_vec = p.ldb % 4 == 0 && aligned16(p.B);
  g.o_vec = splits > 1 ? (p.n % 4 == 0 && aligned16(g.part)) : (p.ldc % 4 == 0 && aligned16(p.C));
  g.m_vec = p.epi == GEMM_MASK && p.ldmask % 4 == 0 && aligned16(p.mask);
  char name[64];
  snprintf(name, sizeof name, "gemm_%s%s_%ldx%ldx%ld", p.ta ? "T" : "N", p.tb ? "T" : "N",
           (long)p.m, (long)p.n, (long)p.k);
  ProfScope prof(name, (int32_t)p.n, p.m, p.k, s);
  gcn_status st;
  if (!p.ta && !p.tb) st = launch_layout<false, false>(g, sh, splits, emu, s);
  else if (!p.ta && p.tb) st = launch_layout<false, true>(g, sh, splits, emu, s);
  else if (p.ta && !p.tb) st = launch_layout<true, false>(g, sh, splits, emu, s);
  else st = launch_layout<true, true>(g, sh, splits, emu, s);
  if (st != GCN_OK || splits == 1) return st;
  return launch_reduce(g.part, splits, p.m, p.n, p.C, p.ldc, p.bias, s);
}

// ---------------------------------------------------------------------------
// column sums (bias gradient) and mean of per-row values (loss), fixed order
// ---------------------------------------------------------------------------
namespace {
constexpr int kColBlocksMax = 1024;

int col_blocks(int64_t rows) { return (int)std::max<int64_t>(1, std::min<int64_t>(kColBlocksMax, ceil_div(rows, 64))); }

// Workgroup b sums rows [b*chunk, (b+1)*chunk).  Thread (c4, rl): columns 4*c4 .. 4*c4+3
// of each 4*CQ-column slab, rows rl, rl + RL, ... (RL = 256 / CQ row lanes); the row
// lanes are combined in lane order.  CQ = 64 for wide matrices; CQ = 16 for at most 64
// columns, where 64 column lanes would leave most threads idle and each busy one a long
// chain of row loads (the loss layer's 40 columns).
template <int CQ>
__global__ void __launch_bounds__(256) k_colsum_partial(int64_t rows, int32_t w, const float* G, int64_t ldg,
                                                        int64_t chunk, const float* rv, double* part,
                                                        int32_t pw, int vec) {
  constexpr int RL = 256 / CQ;
  __shared__ double red[RL][4 * CQ];
  const int c4 = threadIdx.x % CQ, rl = threadIdx.x / CQ;
  const int64_t r0 = (int64_t)blockIdx.x * chunk;
  const int64_t r1 = r0 + chunk < rows ? r0 + chunk : rows;
  for (int cb = 0; cb < w; cb += 4 * CQ) {
    const int c = cb + 4 * c4;
    float a[4] = {0.f, 0.f, 0.f, 0.f}, b[4] = {0.f, 0.f, 0.f, 0.f};
    if (c < w) {
      if (vec && c + 4 <= w) {
        int64_t r = r0 + rl;
        for (; r + RL < r1; r += 2 * RL) {
          const float4 x = *reinterpret_cast<const float4*>(G + r * ldg + c);
          const float4 y = *reinterpret_cast<const float4*>(G + (r + RL) * ldg + c);
          a[0] += x.x; a[1] += x.y; a[2] += x.z; a[3] += x.w;
          b[0] += y.x; b[1] += y.y; b[2] += y.z; b[3] += y.w;
        }
        if (r < r1) {
          const float4 x = *reinterpret_cast<const float4*>(G + r * ldg + c);
          a[0] += x.x; a[1] += x.y; a[2] += x.z; a[3] += x.w;
        }
      } else {
        for (int64_t r = r0 + rl; r < r1; r += RL)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (c + i < w) a[i] += G[r * ldg + c + i];
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) red[rl][4 * c4 + i] = (double)a[i] + (double)b[i];
    __syncthreads();
    if (rl == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (c + i < w) {
          double t = red[0][4 * c4 + i];
#pragma unroll
          for (int q = 1; q < RL; ++q) t += red[q][4 * c4 + i];
          part[(int64_t)blockIdx.x * pw + c + i] = t;
        }
    }
    __syncthreads();
  }
  if (rv) {
    double* flat = &red[0][0];  // 1024 doubles
    double s = 0.0;
    for (int64_t r = r0 + threadIdx.x; r < r1; r += 256) s += (double)rv[r];
    flat[threadIdx.x] = s;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
      if ((int)threadIdx.x < o) flat[threadIdx.x] += flat[threadIdx.x + o];
      __syncthreads();
    }
    if (threadIdx.x == 0) part[(int64_t)blockIdx.x * pw + w] = flat[0];
  }
}

// out[c] = sum_b part[b][c]: 4 columns per workgroup, one wavefront per column; lane q
// sums b = q, q + 64, ... in increasing order into 4 interleaved accumulators (combined
// in order), then the 64 lane sums are combined by a fixed binary tree.
__global__ void __launch_bounds__(256) k_colsum_final(const double* part, int nblk, int32_t w, int32_t pw,
                                                      float* out, float* mean, double inv_rows) {
  __shared__ double red[4][64];
  const int q = threadIdx.x % 64, cl = threadIdx.x / 64;
  const int col = blockIdx.x * 4 + cl;
  double a[4] = {0.0, 0.0, 0.0, 0.0};
  if (col < pw) {
    int b = q;
    for (; b + 192 < nblk; b += 256)
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] += part[(int64_t)(b + 64 * u) * pw + col];
    for (; b < nblk; b += 64) a[0] += part[(int64_t)b * pw + col];
  }
  red[cl][q] = (a[0] + a[1]) + (a[2] + a[3]);
  __syncthreads();
  for (int o = 32; o > 0; o >>= 1) {
    if (q < o) red[cl][q] += red[cl][q + o];
    __syncthreads();
  }
  if (q == 0 && col < pw) {
    const double t = red[cl][0];
    if (col < w) out[col] = (float)t;
    else if (mean) *mean = (float)(t * inv_rows);
  }
}
}  // namespace

size_t colsum_workspace(int64_t rows, int32_t w) {
  return sizeof(double) * (size_t)col_blocks(rows) * (size_t)(w + 1);
}

gcn_status launch_colsum(int64_t rows, int32_t w, const float* G, int64_t ldg, float* out,
                         const float* row_vals, float* mean, void* ws, hipStream_t s) {
  const int32_t pw = w + (row_vals ? 1 : 0);
  if (pw == 0) return GCN_OK;
  const int nblk = col_blocks(rows);
  const int64_t chunk = rows > 0 ? ceil_div(rows, nblk) : 1;
  double* part = static_cast<double*>(ws);
  const int vec = G && ldg % 4 == 0 && aligned16(G);
  if (w <= 64)
    hipLaunchKernelGGL(k_colsum_partial<16>, dim3(nblk), dim3(256), 0, s, rows, w, G, ldg, chunk, row_vals,
                       part, pw, vec);
  else
    hipLaunchKernelGGL(k_colsum_partial<64>, dim3(nblk), dim3(256), 0, s, rows, w, G, ldg, chunk, row_vals,
                       part, pw, vec);
  GCN_TRY(check_launch("column sums"));
  hipLaunchKernelGGL(k_colsum_final, dim3((unsigned)ceil_div(pw, 4)), dim3(256), 0, s, part, nblk, w, pw,
                     out, mean, rows > 0 ? 1.0 / (double)rows : 0.0);
  return check_launch("column sums final");
}

}  // namespace gcn
