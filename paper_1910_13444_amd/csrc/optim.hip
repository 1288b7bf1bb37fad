// Parameter update of the fp32 master weights (the paper keeps a
// single-precision copy of the weights and accumulates the gradients in it,
// Sec. III.C).  The paper names no optimizer; the update is Adam (Kingma and
// Ba, 2015) in its textbook form:
//   m = b1 m + (1 - b1) g,   v = b2 v + (1 - b2) g^2,
//   p = p - lr (m c1) / (sqrt(v c2) + eps),  c1 = 1/(1 - b1^t), c2 = 1/(1 - b2^t).
// A step whose gradients were flagged non-finite by the training step (the
// step's device flag) leaves p, m and v unchanged, decided on the device so
// that the caller need not synchronise before the update.
#include "optim.h"

namespace pigan {

__global__ void __launch_bounds__(256)
k_adam(int64_t n, float* __restrict__ p, const float* __restrict__ g, float* __restrict__ m, float* __restrict__ v,
       float lr, float b1, float b2, float eps, float c1, float c2, const int32_t* __restrict__ skip) {
  if (skip && *skip) return;   // one flag for the whole launch
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const float gi = g[i];
    const float mi = b1 * m[i] + (1.0f - b1) * gi;
    const float vi = b2 * v[i] + (1.0f - b2) * gi * gi;
    m[i] = mi;
    v[i] = vi;
    p[i] -= lr * (mi * c1) / (sqrtf(vi * c2) + eps);
  }
}

hipError_t launch_adam(int64_t n, float* p, const float* g, float* m, float* v, float lr, float b1, float b2,
                       float eps, float c1, float c2, const int32_t* skip, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;   // grid-stride beyond 16 waves per CU
  k_adam<<<(unsigned)blocks, 256, 0, st>>>(n, p, g, m, v, lr, b1, b2, eps, c1, c2, skip);
  return hipGetLastError();
}

}  // namespace pigan
