// static_ws.hip -- gcn_gemm_static: the dense product of gcn_gemm with its scratch in a
// static device array instead of a caller workspace, for callers that cannot allocate
// device memory.
//
// The scratch of a product (split-k partial tiles of A^T B, the split weight planes and
// column-sum partials of the row-panel product) lives in `scratch`, a file-scope device
// array of GCN_STATIC_WS_BYTES.  Each device the library runs on holds its own copy, at
// its own address, until the process ends.  In host code `scratch` names a host-side
// stand-in, not device memory, so the device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and that address is what the kernels
// receive.  Every kernel writes the scratch it later reads, so nothing has to start at
// zero; the array keeps the last call's contents.
#include <mutex>

#include "internal.h"

using gcn::fail;
using gcn::hip_fail;

namespace {

__device__ __align__(256) char scratch[GCN_STATIC_WS_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of this device's `scratch` (looked up on the first call per device).
gcn_status scratch_address(void** out) {
  int dev = -1;
  GCN_HIP(hipGetDevice(&dev), "gcn_gemm_static: hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(GCN_E_UNSUPPORTED, "gcn_gemm_static: device index out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    GCN_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "gcn_gemm_static: hipGetSymbolAddress");
    if (!p) return fail(GCN_E_HIP, "gcn_gemm_static: no device address for the scratch array");
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return GCN_OK;
}

}  // namespace

extern "C" gcn_status gcn_gemm_static(int32_t op, int64_t m, int64_t n, int64_t k, const float* d_A, int64_t lda,
                                      const float* d_B, int64_t ldb, float* d_C, int64_t ldc,
                                      const float* d_bias, int32_t epi, const float* d_mask, int64_t ldmask,
                                      hipStream_t stream) {
  // validation and the scratch size, exactly as gcn_gemm plans the product
  size_t need = 0;
  GCN_TRY(gcn_gemm(op, m, n, k, d_A, lda, d_B, ldb, d_C, ldc, d_bias, epi, d_mask, ldmask, nullptr, &need,
                   stream));
  if (need > (size_t)GCN_STATIC_WS_BYTES)
    return fail(GCN_E_CAPACITY, "gcn_gemm_static: the product needs " + std::to_string(need) +
                                         " bytes of scratch, more than the static " +
                                         std::to_string((long long)GCN_STATIC_WS_BYTES));
  void* ws = nullptr;
  GCN_TRY(scratch_address(&ws));
  size_t have = (size_t)GCN_STATIC_WS_BYTES;
  return gcn_gemm(op, m, n, k, d_A, lda, d_B, ldb, d_C, ldc, d_bias, epi, d_mask, ldmask, ws, &have, stream);
}
