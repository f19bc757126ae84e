// bom_ema kernel: the task-space EMA and its bias correction (Sec. 3.2, Eq. (2); Algorithm 1):
//   q = beta1 q + (1 - beta1) s,   q_hat = q * inv_bc1,   inv_bc1 = 1 / (1 - beta1^t).
// O(V) and launch-latency bound: one thread per element.
#include "common.hpp"
#include "kernels.hpp"

namespace bom {
namespace {

__global__ __launch_bounds__(256) void ema_kernel(float* __restrict__ q, const float* __restrict__ s, int64_t V,
                                                  float beta1, float one_minus_beta1, float inv_bc1,
                                                  float* __restrict__ q_hat) {
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j >= V) return;
    const float qn = beta1 * q[j] + one_minus_beta1 * s[j];
    q[j] = qn;
    q_hat[j] = qn * inv_bc1;
}

}  // namespace

hipError_t launch_ema(float* q, const float* s, int64_t V, float beta1, float inv_bc1, float* q_hat,
                      hipStream_t stream) {
    const float omb = (float)(1.0 - (double)beta1);
    const unsigned grid = (unsigned)((V + 255) / 256);
    hipLaunchKernelGGL(ema_kernel, dim3(grid), dim3(256), 0, stream, q, s, V, beta1, omb, inv_bc1, q_hat);
    return hipGetLastError();
}

}  // namespace bom
