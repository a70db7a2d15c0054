// gemm_rows.hip -- C = A B for a tall A and a small B (n <= 256), bf16x6 arithmetic.
//
// The transform products of a GCN layer multiply an N x k feature matrix by a k x n
// weight (H W forward, Q W^T for the input gradient, Section III-A / Algorithm 1), with N
// in the hundreds of thousands and k, n at most a few hundred.  The general tiled GEMM
// re-splits the weight in every workgroup and reads each row of A once per 128 output
// columns; here instead:
//  * B is split once per call (k_split_b) into three bf16 planes stored in the exact
//    order the matrix-core fragments consume them: block (slab, step, column tile,
//    plane) holds, for lane l, the 8 bf16 of column 32 j + l % 32 at the 8 k positions
//    that lane feeds to v_mfma_f32_32x32x16_bf16 (1 KB per block, one 16-byte read per
//    lane, no bank conflicts);
//  * a wavefront owns 32 rows of C and every output column, so each element of A is
//    loaded from HBM and split exactly once.  A goes straight from global memory into
//    the fragment registers (no LDS, no barrier): within a 32-wide k slab, lane half h
//    of row r loads k = 8 i + 4 h .. + 3 for i = 0..3 (32 contiguous bytes per row and
//    load), and MFMA step t takes the loads i = 2t, 2t+1 -- a fixed permutation of k
//    inside the slab, applied identically to B by the split, which a sum over k does
//    not see;
//  * the four wavefronts of a workgroup (128 rows) share B through LDS one 16-k step at
//    a time, double-buffered: the next step is read from L2 while the current one
//    feeds the matrix cores, with one barrier per step; two workgroups share a CU;
//  * the epilogue (bias, ReLU, or the input-gradient mask as a bitmask) stages the
//    accumulators through LDS and writes C in 256-byte row segments with non-temporal
//    stores; with ReLU it can also write the bitmask 1[C > 0] (one bit per element).
// Products with an fp32 1[mask > 0] epilogue use the tiled kernel of gemm.hip.
// The arithmetic per product is that of gemm.hip's bf16x6 mode (the same six part
// products, fp32 accumulation), summed in a different order.
#include <cstdlib>
#include <cstring>

#include "bf16x6.h"
#include "lanes.h"

namespace gcn {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kRowsPerWave = 32;
constexpr int kRowsPerBlock = kWaves * kRowsPerWave;
constexpr int kSlab = 32;          // k per slab: two 32x32x16 steps
constexpr int kBlockBf16 = 64 * 8;  // one fragment block: 64 lanes x 8 bf16 (1 KB)
constexpr int kStagePitch = 64 + 4;   // floats per staged epilogue row
constexpr int kMaxN = 256;            // output columns served
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Slab-local k of MFMA step t, lane half h, fragment element e (0..7).
__host__ __device__ constexpr int kmap(int t, int h, int e) { return 16 * t + 8 * (e >> 2) + 4 * h + (e & 3); }

struct RowsArgs {
  GemmParams p;
  const __bf16* bp;  // split B: [slab][step][column tile][plane][lane][8]
  int nj;            // column tiles (ceil(n / 32))
  int64_t nslab;
  int c_vec;         // C rows 16-byte aligned with ldc % 4 == 0
  float* part;       // p.colsum: per-workgroup column sums [workgroups][n]
  int groups;        // column groups (1 or 2): workgroups per row panel
  int64_t panels;    // row panels of 128 rows
};

// Thread i of a split of B (k x n, or its transpose stored n x k): 8 values of B for one
// (slab, step, column tile, lane), split into 3 planes.
__device__ __forceinline__ void split_b_one(const float* B, int64_t ldb, bool tb, int64_t kk, int64_t nn, int nj,
                                            int64_t i, __bf16* out) {
  const int l = (int)(i % 64);
  const int64_t blk = i / 64;  // (slab * 2 + t) * nj + j
  const int j = (int)(blk % nj);
  const int64_t st = blk / nj;
  const int t = (int)(st % 2);
  const int64_t s = st / 2;
  const int64_t col = (int64_t)j * 32 + l % 32;
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int64_t k = s * kSlab + kmap(t, l / 32, e);
    v[e] = 0.f;
    if (k < kk && col < nn) v[e] = tb ? B[col * ldb + k] : B[k * ldb + col];
  }
  uint4 hi, mid, lo;
  split_pair(v[0], v[1], hi.x, mid.x, lo.x);
  split_pair(v[2], v[3], hi.y, mid.y, lo.y);
  split_pair(v[4], v[5], hi.z, mid.z, lo.z);
  split_pair(v[6], v[7], hi.w, mid.w, lo.w);
  uint4* o = reinterpret_cast<uint4*>(out + (blk * 3) * kBlockBf16) + l;
  o[0] = hi;
  o[64] = mid;
  o[128] = lo;
}

// Threads of one split: 64 per (slab, step, column tile).
inline int64_t split_threads(int64_t k, int64_t n) { return ceil_div(k, kSlab) * 2 * ceil_div(n, 32) * 64; }

__global__ void __launch_bounds__(256) k_split_b(RowsArgs r, int64_t total, __bf16* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  split_b_one(r.p.B, r.p.ldb, r.p.tb, r.p.k, r.p.n, r.nj, i, out);
}

struct SplitBatch {
  const float* B[kMaxSplitJobs];
  __bf16* out[kMaxSplitJobs];
  int64_t ldb[kMaxSplitJobs], k[kMaxSplitJobs], n[kMaxSplitJobs];
  int64_t first[kMaxSplitJobs + 1];  // first thread of each job
  int32_t tb[kMaxSplitJobs], nj[kMaxSplitJobs];
  int32_t count;
};

// Every job of the batch in one launch; thread i belongs to the job whose range holds it.
__global__ void __launch_bounds__(256) k_split_batch(SplitBatch b) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= b.first[b.count]) return;
  int q = 0;
  while (i >= b.first[q + 1]) ++q;
  split_b_one(b.B[q], b.ldb[q], b.tb[q] != 0, b.k[q], b.n[q], b.nj[q], i - b.first[q], b.out[q]);
}

// Split 8 fp32 (two float4) into the three bf16x8 fragment parts.
__device__ __forceinline__ void split8(const float4& a, const float4& b, bf16x8& hi, bf16x8& mid, bf16x8& lo) {
  uint4 h, m, o;
  split_pair(a.x, a.y, h.x, m.x, o.x);
  split_pair(a.z, a.w, h.y, m.y, o.y);
  split_pair(b.x, b.y, h.z, m.z, o.z);
  split_pair(b.z, b.w, h.w, m.w, o.w);
  hi = __builtin_bit_cast(bf16x8, h);
  mid = __builtin_bit_cast(bf16x8, m);
  lo = __builtin_bit_cast(bf16x8, o);
}

// NJ column tiles of 32; PD slabs of A in flight per wavefront.
// Two wavefronts per SIMD (two workgroups per CU): one workgroup's epilogue and barrier
// waits overlap the other's matrix work.
template <int NJ, int PD, int EPI>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) k_gemm_rows(RowsArgs r) {
  constexpr int kStepBf16 = NJ * 3 * kBlockBf16;  // B of one 16-k step
  constexpr int kChunks = kStepBf16 / 8;          // 16-byte pieces per step
  constexpr int kPer = (kChunks + kThreads - 1) / kThreads;
  // two B steps during the k walk, then the epilogue staging (32 x 68 floats per wave)
  // (+ the wavefronts' column sums of the mask epilogue)
  constexpr int kStageBf16 = 2 * kWaves * kRowsPerWave * kStagePitch + (EPI == GEMM_MASK ? 2 * kWaves * kMaxN : 0);
  constexpr int kLdsBf16 = 2 * kStepBf16 > kStageBf16 ? 2 * kStepBf16 : kStageBf16;
  __shared__ __attribute__((aligned(16))) __bf16 lds[kLdsBf16];

  const GemmParams& p = r.p;
  const int tid = threadIdx.x, l = tid % 64;
  const int wave = __builtin_amdgcn_readfirstlane(tid / 64);  // wave-uniform: scalar registers
  const int h = l / 32, l32 = l % 32;
  // Row panel and column group (tiles jb .. jb + NJ - 1 of the r.nj column tiles).  With
  // two groups, workgroup ids (dealt to the 8 XCDs in turn: id % 8 is the XCD) are mapped
  // so that the two groups of a panel run on one XCD, eight ids apart, and the second
  // reads the panel's rows of A from that XCD's L2.
  int64_t panel = blockIdx.x;
  int grp = 0;
  if (r.groups == 2) {
    const int64_t t = (int64_t)blockIdx.x / 8;
    panel = (t / 2) * 8 + blockIdx.x % 8;
    grp = (int)(t % 2);
    if (panel >= r.panels) return;  // the whole workgroup: no barrier has been reached
  }
  const int64_t row0 = panel * kRowsPerBlock + (int64_t)wave * kRowsPerWave;
  const int jb = grp * NJ;
  const int64_t cb = (int64_t)jb * 32;
  const int64_t nslab = r.nslab, nstep = 2 * nslab;

  // this lane's A row (rows past the end re-read the last row; never stored)
  const int64_t arow = row0 + l32 < p.m ? row0 + l32 : p.m - 1;
  const float* ap = p.A + arow * p.lda + 4 * h;
  const bool kfull = p.k % kSlab == 0;
  auto load_a = [&](int64_t s, float4 (&ra)[4]) __attribute__((always_inline)) {
    const float* q = ap + s * kSlab;
    if (kfull || (s + 1) * kSlab <= p.k) {
#pragma unroll
      for (int i = 0; i < 4; ++i) ra[i] = *reinterpret_cast<const float4*>(q + 8 * i);
    } else {
      // partial last slab: zeros past k (the split B is zero there too)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t k0 = s * kSlab + 8 * i + 4 * h;
        float t4[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) t4[c] = k0 + c < p.k ? q[8 * i + c] : 0.f;
        ra[i] = make_float4(t4[0], t4[1], t4[2], t4[3]);
      }
    }
  };
  const u32x4* bsrc = reinterpret_cast<const u32x4*>(r.bp);
  auto load_b = [&](int64_t g, u32x4 (&rb)[kPer]) __attribute__((always_inline)) {
    const u32x4* q = bsrc + (g * r.nj + jb) * (3 * 64);
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (kChunks % kThreads == 0 || tid + i * kThreads < kChunks) rb[i] = q[tid + i * kThreads];
  };
  auto store_b = [&](int buf, const u32x4 (&rb)[kPer]) __attribute__((always_inline)) {
    u32x4* q = reinterpret_cast<u32x4*>(lds + buf * kStepBf16);
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (kChunks % kThreads == 0 || tid + i * kThreads < kChunks) q[tid + i * kThreads] = rb[i];
  };

  floatx16 acc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.f;

  static_assert(PD >= 1 && PD <= 3, "A slabs in flight: 1 to 3");
  float4 ra[PD][4];
  u32x4 rb[kPer];
  load_a(0, ra[0]);  // nslab >= 1 (k > 0)
  if constexpr (PD > 1)
    if (nslab > 1) load_a(1, ra[1]);
  if constexpr (PD > 2)
    if (nslab > 2) load_a(2, ra[2]);
  load_b(0, rb);
  store_b(0, rb);
  __syncthreads();

  // one MFMA step (16 k) of every column tile with the A parts of this lane's row; two
  // tiles at a time, their accumulation chains interleaved
  auto step = [&](int buf, const bf16x8& ah, const bf16x8& am, const bf16x8& al) __attribute__((always_inline)) {
    const bf16x8* f0 = reinterpret_cast<const bf16x8*>(lds + buf * kStepBf16) + l;
#pragma unroll
    for (int j = 0; j + 1 < NJ; j += 2) {
      const bf16x8* f = f0 + j * 3 * 64;
      const bf16x8 bh0 = f[0], bm0 = f[64], bo0 = f[128], bh1 = f[192], bm1 = f[256], bo1 = f[320];
      acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh0, acc[j], 0, 0, 0);
      acc[j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh1, acc[j + 1], 0, 0, 0);
      acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am, bm0, acc[j], 0, 0, 0);
      acc[j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am, bm1, acc[j + 1], 0, 0, 0);
      acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bo0, acc[j], 0, 0, 0);
      acc[j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bo1, acc[j + 1], 0, 0, 0);
      acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am, bh0, acc[j], 0, 0, 0);
      acc[j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am, bh1, acc[j + 1], 0, 0, 0);
      acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bm0, acc[j], 0, 0, 0);
      acc[j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bm1, acc[j + 1], 0, 0, 0);
      acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh0, acc[j], 0, 0, 0);
      acc[j + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh1, acc[j + 1], 0, 0, 0);
    }
    if constexpr (NJ % 2 == 1) {
      const bf16x8* f = f0 + (NJ - 1) * 3 * 64;
      const bf16x8 bh = f[0], bm = f[64], bo = f[128];
      floatx16& c = acc[NJ - 1];
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bh, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am, bm, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bo, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(am, bh, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bm, c, 0, 0, 0);
      c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bh, c, 0, 0, 0);
    }
  };
  // slab s (steps 2s in LDS buffer 0 and 2s + 1 in buffer 1), whose A values are in cur
  // (refilled with slab s + PD).  The B of the next step is read from L2 while the
  // current step runs; a buffer is rewritten only after the barrier that ends the step
  // which last read it.
  auto slab = [&](int64_t s, float4 (&cur)[4]) __attribute__((always_inline)) {
    if (s >= nslab) return;
    const int64_t g = 2 * s;
    load_b(g + 1, rb);
    bf16x8 ah0, am0, al0, ah1, am1, al1;
    split8(cur[0], cur[1], ah0, am0, al0);
    split8(cur[2], cur[3], ah1, am1, al1);
    if (s + PD < nslab) load_a(s + PD, cur);
    step(0, ah0, am0, al0);
    store_b(1, rb);
    __syncthreads();
    if (g + 2 < nstep) load_b(g + 2, rb);
    step(1, ah1, am1, al1);
    if (g + 2 < nstep) store_b(0, rb);
    __syncthreads();
  };
  for (int64_t s0 = 0; s0 < nslab; s0 += PD) {
    slab(s0, ra[0]);
    if constexpr (PD > 1) slab(s0 + 1, ra[1]);
    if constexpr (PD > 2) slab(s0 + 2, ra[2]);
  }

  // Epilogue, two column tiles (32 rows x 64 columns) at a time per wavefront: the
  // accumulators (lane l32 holds column l32 of rows 8 (e / 4) + 4 h + e % 4) go to this
  // wavefront's part of the LDS, which the B steps no longer use (the last step ended
  // with a barrier), and come back as row-contiguous 16-byte vectors, so that C is written
  // in 256-byte row segments (bias and ReLU apply there).  C is touched once: non-temporal
  // stores keep it from displacing the split B in L2 (measured: 20 % faster on the
  // 169,343 x 256 x 256 product).
  float* stage = reinterpret_cast<float*>(lds) + wave * kRowsPerWave * kStagePitch;
  const int sr = l / 16, sc = 4 * (l % 16);  // read-back: rows sr + 4 i, columns sc .. sc + 3
  // Every bias value and mask word the epilogue uses, requested before its first store:
  // one counter tracks a wavefront's loads and stores alike, so a wait for a load issued
  // between stores also waits for those stores, and loads inside the store loop would
  // serialise it on store completion.
  constexpr int kPairs = (NJ + 1) / 2;
  // this workgroup's columns end at ce (a pair may run past a group's last tile)
  const int64_t ce = cb + NJ * 32 < p.n ? cb + NJ * 32 : p.n;
  float bias_all[kPairs][4];
  uint32_t mask_all[kPairs][EPI == GEMM_MASK ? 8 : 1];
#pragma unroll
  for (int jp = 0; jp < kPairs; ++jp) {
    const int64_t col = cb + (int64_t)jp * 64 + sc;
    const bool cin = col < ce;
#pragma unroll
    for (int q = 0; q < 4; ++q) bias_all[jp][q] = p.bias && cin && col + q < ce ? p.bias[col + q] : 0.f;
    if constexpr (EPI == GEMM_MASK) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int64_t row = row0 + sr + 4 * i;
        mask_all[jp][i] = row < p.m && cin ? p.mask_bits[row * p.ld_mask_bits + col / 32] : 0u;
      }
    }
  }
  // Wait for them here, once: the compiler cannot prove them complete across the
  // per-row branches below and would otherwise wait again (for every store so far) at
  // each use.  s_waitcnt vmcnt(0), expcnt and lgkmcnt not waited for.
  __builtin_amdgcn_s_waitcnt(0xF70);
#pragma unroll
  for (int j0 = 0; j0 < NJ; j0 += 2) {
#pragma unroll
    for (int jj = 0; jj < 2 && j0 + jj < NJ; ++jj)
#pragma unroll
      for (int e = 0; e < 16; ++e) stage[(8 * (e / 4) + 4 * h + e % 4) * kStagePitch + 32 * jj + l32] = acc[j0 + jj][e];
    // the wavefront's own staging area: LDS accesses of one wavefront complete in order,
    // the fence keeps the compiler from reordering them
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    const int64_t col = cb + (int64_t)j0 * 32 + sc;
    const bool cin = col < ce, full = col + 4 <= ce;
    const float* bias = bias_all[j0 / 2];
    // bitmask words: 8 lanes (32 columns) per word; the lanes of a word share the row
    const int64_t word = col / 32;
    const int shift = (int)(col % 32);
    float cs[4] = {0.f, 0.f, 0.f, 0.f};  // column sums of this lane's rows (mask epilogue)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t row = row0 + sr + 4 * i;
      const bool rin = row < p.m;  // uniform over the 16 lanes of a row
      const float4 t = *reinterpret_cast<const float4*>(stage + (sr + 4 * i) * kStagePitch + sc);
      float v[4] = {t.x + bias[0], t.y + bias[1], t.z + bias[2], t.w + bias[3]};
      if constexpr (EPI == GEMM_RELU) {
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = fmaxf(v[q], 0.f);
        if (p.relu_bits) {
          uint32_t bits = 0;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (col + q < ce && v[q] > 0.f) bits |= 1u << (shift + q);
          bits = group_or<8>(bits);
          if (rin && cin && l % 8 == 0) p.relu_bits[row * p.ld_relu_bits + word] = bits;
        }
      }
      if constexpr (EPI == GEMM_MASK) {
        const uint32_t mw = mask_all[j0 / 2][i] >> shift;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[q] = (mw >> q) & 1u ? v[q] : 0.f;
          cs[q] += v[q];  // rows past m have mw = 0
        }
      }
      if (!rin || !cin) continue;
      float* cp = p.C + row * p.ldc + col;
      if (full && r.c_vec) {
        const f32x4 o = {v[0], v[1], v[2], v[3]};
        __builtin_nontemporal_store(o, reinterpret_cast<f32x4*>(cp));
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (col + q < ce) cp[q] = v[q];
      }
    }
    if constexpr (EPI == GEMM_MASK) {
      if (r.part) {
        // the four lanes of a column (rows sr = 0..3) in a fixed order, then one partial
        // row of this wavefront's 32 rows
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          cs[q] += __shfl_xor(cs[q], 16, 64);
          cs[q] += __shfl_xor(cs[q], 32, 64);
        }
        float* ws = reinterpret_cast<float*>(lds) + kWaves * kRowsPerWave * kStagePitch + wave * kMaxN + col;
        if (sr == 0 && cin)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (col + q < ce) ws[q] = cs[q];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");  // before the next pair's writes
  }
  if constexpr (EPI == GEMM_MASK) {
    if (r.part) {
      // the workgroup's partial row: the wavefronts' sums of column t, in wavefront order
      __syncthreads();
      const float* ws = reinterpret_cast<const float*>(lds) + kWaves * kRowsPerWave * kStagePitch;
      for (int64_t t = cb + tid; t < ce; t += kThreads) {
        float v = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) v += ws[w * kMaxN + t];
        r.part[panel * p.n + t] = v;
      }
    }
  }
}

template <int NJ, int PD>
void launch_nj(const RowsArgs& r, hipStream_t s) {
  const dim3 grid((unsigned)(r.groups == 2 ? ceil_div(r.panels, 8) * 16 : r.panels));
  switch (r.p.epi) {
    case GEMM_RELU: hipLaunchKernelGGL((k_gemm_rows<NJ, PD, GEMM_RELU>), grid, dim3(kThreads), 0, s, r); break;
    case GEMM_MASK: hipLaunchKernelGGL((k_gemm_rows<NJ, PD, GEMM_MASK>), grid, dim3(kThreads), 0, s, r); break;
    default: hipLaunchKernelGGL((k_gemm_rows<NJ, PD, GEMM_NONE>), grid, dim3(kThreads), 0, s, r);
  }
}

int64_t split_b_elems(const GemmParams& p) {
  return ceil_div(p.k, kSlab) * 2 * ceil_div(p.n, 32) * 3 * kBlockBf16;
}

// Partial rows of the fused column sums: one per workgroup.
int64_t colsum_parts(const GemmParams& p) {
  return p.colsum && p.epi == GEMM_MASK ? ceil_div(p.m, kRowsPerBlock) : 0;
}

}  // namespace

// Below this many rows the extra launch of the weight split costs more than the
// row-panel kernel saves (a Cora-sized epoch is launch-latency bound).
constexpr int64_t kRowsAuto = 32768;

// GCN_GEMM_ROWS=0 sends these products to the general tiled kernel, =1 takes the
// row-panel kernel whatever the row count; unset: from kRowsAuto rows on.
static bool rows_enabled(int64_t m) {
  const char* e = getenv("GCN_GEMM_ROWS");
  if (e && strcmp(e, "0") == 0) return false;
  if (e && strcmp(e, "1") == 0) return true;
  return m >= kRowsAuto;
}

// The mask epilogue runs here only in its bitmask form: with an fp32 mask (a 4-byte read
// per output) the tiled kernel was measured faster on the arxiv-like shapes.
bool gemm_rows_supported(const GemmParams& p) {
  return gemm_bf16x6_mode() && rows_enabled(p.m) && (p.epi != GEMM_MASK || p.mask_bits) && !p.ta && p.n > 0 && p.n <= 256 && p.k > 0 && p.m >= kRowsPerBlock &&
         p.lda % 4 == 0 && aligned16(p.A);
}

size_t gemm_rows_workspace(const GemmParams& p) {
  if (!gemm_rows_supported(p)) return 0;
  const int64_t parts = colsum_parts(p);
  return (size_t)round_up((int64_t)sizeof(__bf16) * split_b_elems(p), 256) +
         (size_t)round_up((int64_t)sizeof(float) * parts * p.n, 256) +
         (parts ? colsum_workspace(parts, (int32_t)p.n) : 0);
}

gcn_status launch_gemm_rows(const GemmParams& p, void* ws, hipStream_t s) {
  RowsArgs r{};
  r.p = p;
  r.nj = (int)ceil_div(p.n, 32);
  r.nslab = ceil_div(p.k, kSlab);
  r.bp = p.bsplit ? static_cast<const __bf16*>(p.bsplit) : static_cast<const __bf16*>(ws);
  r.c_vec = p.ldc % 4 == 0 && aligned16(p.C);
  const int64_t nparts = colsum_parts(p);
  r.part = nparts ? reinterpret_cast<float*>(static_cast<char*>(ws) +
                                             round_up((int64_t)sizeof(__bf16) * split_b_elems(p), 256))
                  : nullptr;
  if (!p.bsplit) {
    const int64_t threads = split_threads(p.k, p.n);
    hipLaunchKernelGGL(k_split_b, dim3((unsigned)ceil_div(threads, 256)), dim3(256), 0, s, r, threads,
                       static_cast<__bf16*>(ws));
    GCN_TRY(check_launch("gemm weight split"));
  }
  // With fewer than 2048 row panels (8 per CU) the last wave of workgroups leaves CUs
  // idle, and with a short k the epilogue (every column of 32 rows per wavefront)
  // dominates.  There the 8 column tiles go to two workgroups of 4 each: half the
  // accumulators per wavefront and twice the workgroups, the second reading the panel's
  // rows of A from L2.  Measured on the arxiv-like products (169,343 rows, 1,323 panels):
  // width-40 input gradient 81.2 -> 72.3 us, 128 -> 256 transform 107 -> 100 us, masked
  // 256 x 256 input gradient 153 -> 149 us, 256 x 256 transform 135.5 -> 138 us; epoch
  // 2.179 -> 2.153 ms.  At 2,449,029 rows (19,133 panels) the width-47 input gradient
  // measured 0.80 -> 0.82 ms, so not there.  GCN_ROWS_GROUPS=1 / =2 force one / two.
  const char* ge = getenv("GCN_ROWS_GROUPS");
  r.panels = ceil_div(p.m, kRowsPerBlock);
  const bool grouped = r.nj == 8 && !(ge && strcmp(ge, "1") == 0) &&
                       (r.panels < 2048 || (ge && strcmp(ge, "2") == 0));
  r.groups = grouped ? 2 : 1;
  if (grouped) launch_nj<4, 2>(r, s);
  else switch (r.nj) {
    case 1: launch_nj<1, 3>(r, s); break;
    case 2: launch_nj<2, 3>(r, s); break;
    case 3: launch_nj<3, 2>(r, s); break;
    case 4: launch_nj<4, 2>(r, s); break;
    case 5: launch_nj<5, 2>(r, s); break;
    case 6: launch_nj<6, 1>(r, s); break;
    case 7: launch_nj<7, 1>(r, s); break;
    default: launch_nj<8, 1>(r, s);
  }
  GCN_TRY(check_launch("gemm (row panels)"));
  if (!nparts) return GCN_OK;
  // the partial rows are a small matrix: its column sums by the two-level fixed-order pass
  void* cws = reinterpret_cast<char*>(r.part) + round_up((int64_t)sizeof(float) * nparts * p.n, 256);
  return launch_colsum(nparts, (int32_t)p.n, r.part, p.n, p.colsum, nullptr, nullptr, cws, s);
}

size_t gemm_rows_split_bytes(const SplitJob& j) {
  return (size_t)round_up((int64_t)sizeof(__bf16) * ceil_div(j.k, kSlab) * 2 * ceil_div(j.n, 32) * 3 * kBlockBf16,
                          256);
}

gcn_status launch_split_batch(const SplitJob* jobs, int count, hipStream_t s) {
  if (count <= 0) return GCN_OK;
  if (count > kMaxSplitJobs) return fail(GCN_E_UNSUPPORTED, "weight split: too many jobs");
  SplitBatch b{};
  b.count = count;
  b.first[0] = 0;
  for (int q = 0; q < count; ++q) {
    const SplitJob& j = jobs[q];
    if (j.k <= 0 || j.n <= 0 || j.n > kMaxN || !j.B || !j.out || !aligned16(j.out))
      return fail(GCN_E_INVALID, "weight split: bad job");
    b.B[q] = j.B;
    b.out[q] = static_cast<__bf16*>(j.out);
    b.ldb[q] = j.ldb;
    b.k[q] = j.k;
    b.n[q] = j.n;
    b.tb[q] = j.tb ? 1 : 0;
    b.nj[q] = (int32_t)ceil_div(j.n, 32);
    b.first[q + 1] = b.first[q] + split_threads(j.k, j.n);
  }
  ProfScope prof("weight_split", 0, 0, 0, s);
  hipLaunchKernelGGL(k_split_batch, dim3((unsigned)ceil_div(b.first[count], 256)), dim3(256), 0, s, b);
  return check_launch("weight split batch");
}

}  // namespace gcn
