// Matrix-core rate probes for the roofline figures of the prefill GEMM and
// of the many-token decode product: the instruction's sustained rate on this
// GPU at the clock it holds under that load, next to the nominal peak.
// Every wave issues eight independent 16 x 16 MFMAs (four 32 x 32) per
// iteration (no memory traffic inside the loop) and writes one word of
// their sums at the end, so none of the work can be dropped.
#include "common.h"

namespace fairy2i {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 256;
constexpr int kProbeChains = 8;  // independent accumulators per wave

// v_mfma_i32_16x16x64_i8: 2 x 16 x 16 x 64 = 32768 operations.
__global__ __launch_bounds__(kProbeThreads) void probe_mfma_i8_kernel(int iters, int32_t* __restrict__ sink) {
  const int t = (int)threadIdx.x;
  const v4i a = v4i{t, t + 1, t + 2, t + 3}, b = v4i{3 * t, t ^ 5, t + 7, 11};
  v4i acc[kProbeChains];
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) acc[j] = v4i{j, 0, 0, 0};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < kProbeChains; ++j) acc[j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc[j], 0, 0, 0);
  }
  int s = 0;
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  sink[(int64_t)blockIdx.x * kProbeThreads + t] = s;
}

// v_mfma_i32_32x32x32_i8: 2 x 32 x 32 x 32 = 65536 operations (four
// accumulators of 16 registers).
__global__ __launch_bounds__(kProbeThreads) void probe_mfma_i8_32_kernel(int iters, int32_t* __restrict__ sink) {
  typedef int v16i __attribute__((ext_vector_type(16)));
  const int t = (int)threadIdx.x;
  const v4i a = v4i{t, t + 1, t + 2, t + 3}, b = v4i{3 * t, t ^ 5, t + 7, 11};
  v16i acc[kProbeChains / 2];
#pragma unroll
  for (int j = 0; j < kProbeChains / 2; ++j) {
    acc[j] = v16i{};
    acc[j][0] = j;
  }
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < kProbeChains / 2; ++j) acc[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[j], 0, 0, 0);
  }
  int s = 0;
#pragma unroll
  for (int j = 0; j < kProbeChains / 2; ++j) s += acc[j][0] + acc[j][15];
  sink[(int64_t)blockIdx.x * kProbeThreads + t] = s;
}

// v_mfma_scale_f32_16x16x128_f8f6f4 with e4m3 (A) and e2m1 (B) operands, the
// decode product's instruction: 2 x 16 x 16 x 128 = 65536 operations.
__global__ __launch_bounds__(kProbeThreads) void probe_mfma_f8f4_kernel(int iters, int32_t* __restrict__ sink) {
  const int t = (int)threadIdx.x;
  const int w = 0x38383838 ^ (t & 0x07070707);  // e4m3 values near 1
  const v8i a = v8i{w, w, w, w, w, w, w, w};
  const int c4 = 0x22222222 | (t & 0x88888888);  // e2m1 +-1
  const v8i b = v8i{c4, c4, c4, c4, 0, 0, 0, 0};
  v4f acc[kProbeChains];
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) acc[j] = v4f{(float)j, 0.f, 0.f, 0.f};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < kProbeChains; ++j)
      acc[j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc[j], 0, 4, 0, 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < kProbeChains; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
  sink[(int64_t)blockIdx.x * kProbeThreads + t] = __float_as_int(s);
}

}  // namespace

}  // namespace fairy2i

using namespace fairy2i;

extern "C" {

fairy2i_status fairy2i_probe_mfma(int32_t kind, int32_t blocks, int32_t iters, int32_t* sink, double* ops,
                                  void* stream) {
  if (!sink || !ops) return FAIRY2I_ERR_NULL;
  if (kind != FAIRY2I_PROBE_MFMA_I8 && kind != FAIRY2I_PROBE_MFMA_F8F4 && kind != FAIRY2I_PROBE_MFMA_I8_32X32)
    return FAIRY2I_ERR_UNSUPPORTED;
  if (blocks < 1 || blocks > (1 << 20) || iters < 1 || iters > (1 << 24)) return FAIRY2I_ERR_SHAPE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  // operations per wave and iteration: eight 16 x 16 MFMAs or four 32 x 32 ones
  const double per = kind == FAIRY2I_PROBE_MFMA_I8 ? 8 * 32768.0 : (kind == FAIRY2I_PROBE_MFMA_F8F4 ? 8 * 65536.0
                                                                                                   : 4 * 65536.0);
  *ops = (double)blocks * (kProbeThreads / 64) * (double)iters * per;
  if (kind == FAIRY2I_PROBE_MFMA_I8)
    hipLaunchKernelGGL(probe_mfma_i8_kernel, dim3((unsigned)blocks), dim3(kProbeThreads), 0, s, iters, sink);
  else if (kind == FAIRY2I_PROBE_MFMA_F8F4)
    hipLaunchKernelGGL(probe_mfma_f8f4_kernel, dim3((unsigned)blocks), dim3(kProbeThreads), 0, s, iters, sink);
  else
    hipLaunchKernelGGL(probe_mfma_i8_32_kernel, dim3((unsigned)blocks), dim3(kProbeThreads), 0, s, iters, sink);
  return hipGetLastError() == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP;
}

}  // extern "C"
