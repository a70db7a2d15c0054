// device_gen.hip -- the input generators' counter stream on the GPU (libsynth.so).
//
// Fills feature matrices directly in device memory with exactly the values the
// numpy generators in gcn_synth/__init__.py produce: entry e of the (seed,
// stream) sequence is the SplitMix64 finaliser (Steele, Lea and Flood, OOPSLA
// 2014) applied to state + (e + 1) * GAMMA.  Used for inputs too large to draw
// on the host (a 2^21 x 4096 matrix is 34 GB); any row range can be redrawn on
// the CPU for checking.  Holds no arithmetic of the GCN method.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// X[r, c] for rows [row0, row0 + rows): entry index e = (row0 + r) * f + c.
// present iff (h >> 32) < thr; value 1 (binary) or (low 24 bits + 1) * 2^-24.
__global__ void k_bernoulli(float* X, int64_t rows, int32_t f, int64_t ldx, int64_t row0, uint64_t state,
                            uint64_t thr, int binary) {
  const int64_t total = rows * (int64_t)f;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / f;
    const int32_t c = (int32_t)(i - r * f);
    const uint64_t e = (uint64_t)(row0 + r) * (uint64_t)f + (uint64_t)c;
    const uint64_t h = mix64(state + (e + 1) * kGamma);
    float v = 0.f;
    if ((h >> 32) < thr) v = binary ? 1.f : (float)((h & 0xFFFFFFull) + 1ull) * (1.f / 16777216.f);
    X[r * ldx + c] = v;
  }
}

}  // namespace

extern "C" {

// Returns 0 on success, the HIP error code otherwise.  `state` is the sequence's
// starting state and `thr` = min(round(p * 2^32), 2^32), both computed by the caller.
int synth_bernoulli(float* d_X, int64_t rows, int32_t f, int64_t ldx, int64_t row0, uint64_t state,
                    uint64_t thr, int32_t binary, hipStream_t stream) {
  if (rows <= 0 || f <= 0) return 0;
  const int64_t total = rows * (int64_t)f;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_bernoulli, dim3((unsigned)blocks), dim3(256), 0, stream, d_X, rows, f, ldx, row0,
                     state, thr, binary);
  return (int)hipGetLastError();
}

}  // extern "C"
