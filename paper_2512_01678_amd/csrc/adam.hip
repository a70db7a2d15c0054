// adam.hip -- one fused Adam step over every parameter tensor of the model.
//
// Listing 1 ends each epoch with an Adam step (learning rate 0.01, first- and
// second-moment decay 0.9 and 0.999); the update is the bias-corrected Adam rule
//   m = b1 m + (1-b1) g,  v = b2 v + (1-b2) g^2,
//   p = p - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps),
// applied elementwise.  All tensors go in one launch (their pointers travel
// in the kernel arguments), so the step costs one launch per epoch.
#include "internal.h"

namespace gcn {
namespace {

constexpr int kMaxTensors = 16;

struct AdamArgs {
  float* p[kMaxTensors];
  const float* g[kMaxTensors];
  float* m[kMaxTensors];
  float* v[kMaxTensors];
  int64_t off[kMaxTensors + 1];
  int32_t count;
  float lr, b1, omb1, b2, omb2, eps, bc1, bc2;  // omb = 1 - b, formed in double
  const int32_t* d_step;                        // when set: bc1, bc2 from 1 - b^(*d_step + 1)
  double b1d, b2d;
};

__global__ void __launch_bounds__(256) k_adam(AdamArgs a) {
  const int64_t total = a.off[a.count];
  // locals, not writes into the argument block: a written argument struct that is also
  // indexed by tensor would be copied to per-lane scratch memory
  float bc1 = a.bc1, bc2 = a.bc2;
  if (a.d_step) {
    const double t = (double)(*a.d_step + 1);
    bc1 = (float)(1.0 - pow(a.b1d, t));
    bc2 = (float)(1.0 - pow(a.b2d, t));
  }
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    int t = 0;
    while (i >= a.off[t + 1]) ++t;
    const int64_t j = i - a.off[t];
    const float g = a.g[t][j];
    const float m = a.b1 * a.m[t][j] + a.omb1 * g;
    const float v = a.b2 * a.v[t][j] + a.omb2 * (g * g);
    a.m[t][j] = m;
    a.v[t][j] = v;
    const float mhat = m / bc1;
    const float vhat = v / bc2;
    a.p[t][j] -= a.lr * mhat / (sqrtf(vhat) + a.eps);
  }
}

__global__ void k_step_increment(int32_t* d_step) {
  if (threadIdx.x == 0) *d_step += 1;
}

}  // namespace

gcn_status launch_adam(const gcn_adam_tensor* t, int32_t count, int32_t step, int32_t* d_step, double lr,
                       double b1, double b2, double eps, hipStream_t s) {
  if (count > kMaxTensors) return fail(GCN_E_UNSUPPORTED, "gcn_adam: at most 16 tensors per call");
  AdamArgs a{};
  a.count = count;
  a.off[0] = 0;
  for (int i = 0; i < count; ++i) {
    a.p[i] = t[i].param;
    a.g[i] = t[i].grad;
    a.m[i] = t[i].m;
    a.v[i] = t[i].v;
    a.off[i + 1] = a.off[i] + t[i].count;
  }
  a.lr = (float)lr;
  a.b1 = (float)b1;
  a.omb1 = (float)(1.0 - b1);
  a.b2 = (float)b2;
  a.omb2 = (float)(1.0 - b2);
  a.eps = (float)eps;
  a.bc1 = (float)(1.0 - std::pow(b1, (double)step));
  a.bc2 = (float)(1.0 - std::pow(b2, (double)step));
  a.d_step = d_step;
  a.b1d = b1;
  a.b2d = b2;
  const int64_t total = a.off[count];
  if (total > 0) {
    const unsigned grid = (unsigned)std::min<int64_t>(ceil_div(total, 256), 2048);
    hipLaunchKernelGGL(k_adam, dim3(grid), dim3(256), 0, s, a);
    GCN_TRY(check_launch("adam"));
  }
  if (d_step) {
    hipLaunchKernelGGL(k_step_increment, dim3(1), dim3(64), 0, s, d_step);
    GCN_TRY(check_launch("adam step"));
  }
  return GCN_OK;
}

}  // namespace gcn
