// Per-token int8 activations: absmax over the 2K real components of a token,
// q = clamp(rint(x * (127 / g)), -127, 127), dequantisation factor g / 127,
// all in float32 with IEEE division (no fast-math).  One block per token;
// the absmax is a max, so its value does not depend on reduction order.
#include "common.h"

namespace fairy2i {

namespace {

template <int DT>
__device__ inline float load_act(const void* x, int64_t i) {
  if constexpr (DT == FAIRY2I_ACT_F32) {
    return static_cast<const float*>(x)[i];
  } else {
    const uint32_t bits = static_cast<const uint16_t*>(x)[i];
    return __uint_as_float(bits << 16);
  }
}

template <int DT>
__global__ __launch_bounds__(256) void act_quant_kernel(const void* __restrict__ x, int64_t K,
                                                        int8_t* __restrict__ q,
                                                        float* __restrict__ x_scale) {
  __shared__ float red[256 / 64];
  const int64_t b = blockIdx.x;
  const int64_t n = 2 * K;
  const int64_t base = b * n;
  float m = 0.0f;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) m = fmaxf(m, fabsf(load_act<DT>(x, base + i)));
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  float g = red[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) g = fmaxf(g, red[w]);
  if (g == 0.0f) {
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) q[base + i] = 0;
    if (threadIdx.x == 0) x_scale[b] = 0.0f;
    return;
  }
  const float inv = 127.0f / g;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
    const float v = __fmul_rn(load_act<DT>(x, base + i), inv);
    float r = rintf(v);
    r = fminf(fmaxf(r, -127.0f), 127.0f);
    q[base + i] = (int8_t)(int)r;
  }
  if (threadIdx.x == 0) x_scale[b] = g / 127.0f;
}

}  // namespace

hipError_t launch_quantize_act_int8(const void* x, int dtype, int64_t B, int64_t K, int8_t* q,
                                    float* x_scale, hipStream_t stream) {
  if (dtype == FAIRY2I_ACT_F32)
    hipLaunchKernelGGL(act_quant_kernel<FAIRY2I_ACT_F32>, dim3((unsigned)B), dim3(256), 0, stream, x,
                       K, q, x_scale);
  else
    hipLaunchKernelGGL(act_quant_kernel<FAIRY2I_ACT_BF16>, dim3((unsigned)B), dim3(256), 0, stream, x,
                       K, q, x_scale);
  return hipGetLastError();
}

}  // namespace fairy2i
