// Real layer -> widely-linear pair (Sec. 3.1, Eq. UW-from-R).
//
// One thread per complex entry (i, j).  The four real blocks are read at
// A[i][j], A[i][K+j], A[N+i][j], A[N+i][K+j]; consecutive threads take
// consecutive j, so every load and store is coalesced.  The half-sums are
// formed in double (exact for float operands) and rounded once to float.
#include "common.h"

namespace fairy2i {

__global__ __launch_bounds__(256) void to_wl_kernel(const float* __restrict__ A, int64_t N,
                                                    int64_t K, float2* __restrict__ U,
                                                    float2* __restrict__ W) {
  const int64_t total = N * K;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
    const int64_t i = idx / K, j = idx - (idx / K) * K;
    const float* top = A + i * 2 * K;
    const float* bot = A + (N + i) * 2 * K;
    const double r11 = top[j], r12 = top[K + j], r21 = bot[j], r22 = bot[K + j];
    U[idx] = make_float2((float)(0.5 * (r11 + r22)), (float)(0.5 * (r21 - r12)));
    W[idx] = make_float2((float)(0.5 * (r11 - r22)), (float)(0.5 * (r12 + r21)));
  }
}

hipError_t launch_to_widely_linear(const float* A, int64_t N, int64_t K, float2* U, float2* W,
                                   hipStream_t stream) {
  const int64_t total = N * K;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(to_wl_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, A, N, K, U, W);
  return hipGetLastError();
}

}  // namespace fairy2i
