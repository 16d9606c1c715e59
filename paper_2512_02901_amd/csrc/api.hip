// C-ABI entry points: argument checks on the host, then launches on the
// caller's stream.  Nothing here allocates, frees or synchronises.
#include <stddef.h>

#include <vector>

#include "common.h"
#include "superacc.h"

using namespace fairy2i;

namespace {

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

inline fairy2i_status hip_status(hipError_t e) { return e == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP; }

fairy2i_status check_wl_common(const uint8_t* cu, const uint8_t* cw, int32_t T, int64_t N, int64_t K,
                               const void* x, int64_t B, const void* out) {
  if (!cu || !cw || !x || !out) return FAIRY2I_ERR_NULL;
  if (N <= 0 || K <= 0 || B <= 0 || (K % 4) != 0) return FAIRY2I_ERR_SHAPE;
  // int32 accumulators: |sum| <= 127 K must stay below 2^31; grid limits.
  if (K > ((int64_t)1 << 24) || N > ((int64_t)1 << 31) - 64 || B > ((int64_t)1 << 31) - 64)
    return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  return FAIRY2I_OK;
}

}  // namespace

extern "C" {

const char* fairy2i_status_string(fairy2i_status s) {
  switch (s) {
    case FAIRY2I_OK: return "ok";
    case FAIRY2I_ERR_NULL: return "null pointer argument";
    case FAIRY2I_ERR_SHAPE: return "dimension out of range";
    case FAIRY2I_ERR_STAGES: return "number of stages T out of range";
    case FAIRY2I_ERR_DTYPE: return "unknown activation dtype";
    case FAIRY2I_ERR_UNSUPPORTED: return "unsupported argument combination";
    case FAIRY2I_ERR_WORKSPACE: return "workspace missing or too small";
    case FAIRY2I_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int32_t fairy2i_abi_version(void) { return 1; }

fairy2i_status fairy2i_to_widely_linear(const float* A, int64_t rows, int64_t cols, float* U,
                                        float* W, void* stream) {
  if (!A || !U || !W) return FAIRY2I_ERR_NULL;
  if (rows <= 0 || cols <= 0 || (rows % 2) != 0 || (cols % 2) != 0) return FAIRY2I_ERR_SHAPE;
  return hip_status(launch_to_widely_linear(A, rows / 2, cols / 2, reinterpret_cast<float2*>(U),
                                            reinterpret_cast<float2*>(W), as_stream(stream)));
}

size_t fairy2i_quantize_workspace_bytes(int64_t N, int64_t K, int32_t T) {
  (void)T;
  if (N <= 0 || K <= 0) return 0;
  return quantize_workspace_bytes(N, K);
}

fairy2i_status fairy2i_quantize(const float* M, int64_t N, int64_t K, int32_t T, uint8_t* codes,
                                float* scales, void* workspace, size_t workspace_bytes, void* stream) {
  if (!M || !codes || !scales) return FAIRY2I_ERR_NULL;
  if (N <= 0 || K <= 0 || (K % 4) != 0 || N > FAIRY2I_MAX_QUANTIZE_ENTRIES / K)
    return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (!workspace || workspace_bytes < quantize_workspace_bytes(N, K)) return FAIRY2I_ERR_WORKSPACE;
  return hip_status(launch_quantize(reinterpret_cast<const float2*>(M), N, K, T, codes, scales,
                                    workspace, as_stream(stream)));
}

fairy2i_status fairy2i_quantize_act_int8(const void* x, int32_t dtype, int64_t B, int64_t K,
                                         int8_t* q, float* x_scale, void* stream) {
  if (!x || !q || !x_scale) return FAIRY2I_ERR_NULL;
  if (B <= 0 || K <= 0 || B > ((int64_t)1 << 31) - 1) return FAIRY2I_ERR_SHAPE;
  if (dtype != FAIRY2I_ACT_F32 && dtype != FAIRY2I_ACT_BF16) return FAIRY2I_ERR_DTYPE;
  return hip_status(launch_quantize_act_int8(x, dtype, B, K, q, x_scale, as_stream(stream)));
}

size_t fairy2i_wl_matmul_workspace_bytes(int64_t N, int64_t K, int32_t T, int64_t B, int32_t dtype) {
  (void)N; (void)K; (void)T; (void)B; (void)dtype;
  return 0;
}

fairy2i_status fairy2i_wl_matmul(const uint8_t* codes_U, const float* scales_U,
                                 const uint8_t* codes_W, const float* scales_W, int32_t T,
                                 int64_t N, int64_t K, const void* x, const float* x_scale,
                                 int32_t dtype, int64_t B, float* y, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  fairy2i_status st = check_wl_common(codes_U, codes_W, T, N, K, x, B, y);
  if (st != FAIRY2I_OK) return st;
  if (!scales_U || !scales_W) return FAIRY2I_ERR_NULL;
  if (dtype != FAIRY2I_ACT_F32 && dtype != FAIRY2I_ACT_BF16 && dtype != FAIRY2I_ACT_I8)
    return FAIRY2I_ERR_DTYPE;
  if (dtype == FAIRY2I_ACT_I8 && !x_scale) return FAIRY2I_ERR_NULL;
  if (dtype != FAIRY2I_ACT_I8 && x_scale) return FAIRY2I_ERR_UNSUPPORTED;
  if (dtype != FAIRY2I_ACT_I8 && B > FAIRY2I_MAX_DECODE_BATCH) return FAIRY2I_ERR_UNSUPPORTED;
  if (workspace_bytes < fairy2i_wl_matmul_workspace_bytes(N, K, T, B, dtype) ||
      (fairy2i_wl_matmul_workspace_bytes(N, K, T, B, dtype) > 0 && !workspace))
    return FAIRY2I_ERR_WORKSPACE;
  WlArgs a{};
  a.codes[0] = codes_U;
  a.codes[1] = codes_W;
  a.scales[0] = scales_U;
  a.scales[1] = scales_W;
  a.T = T;
  a.N = N;
  a.K = K;
  a.B = B;
  a.x = x;
  a.x_scale = x_scale;
  a.dtype = dtype;
  a.y = reinterpret_cast<float2*>(y);
  a.acc = nullptr;
  const hipError_t e = (B <= FAIRY2I_MAX_DECODE_BATCH) ? launch_gemv(a, as_stream(stream))
                                                       : launch_gemm_i8(a, as_stream(stream));
  return hip_status(e);
}

fairy2i_status fairy2i_wl_int8_accumulators(const uint8_t* codes_U, const uint8_t* codes_W, int32_t T,
                                            int64_t N, int64_t K, const int8_t* q, int64_t B,
                                            int32_t* acc, void* workspace, size_t workspace_bytes,
                                            void* stream) {
  fairy2i_status st = check_wl_common(codes_U, codes_W, T, N, K, q, B, acc);
  if (st != FAIRY2I_OK) return st;
  if (workspace_bytes < fairy2i_wl_matmul_workspace_bytes(N, K, T, B, FAIRY2I_ACT_I8) ||
      (fairy2i_wl_matmul_workspace_bytes(N, K, T, B, FAIRY2I_ACT_I8) > 0 && !workspace))
    return FAIRY2I_ERR_WORKSPACE;
  WlArgs a{};
  a.codes[0] = codes_U;
  a.codes[1] = codes_W;
  a.T = T;
  a.N = N;
  a.K = K;
  a.B = B;
  a.x = q;
  a.dtype = FAIRY2I_ACT_I8;
  a.acc = acc;
  const hipError_t e = (B <= FAIRY2I_MAX_DECODE_BATCH) ? launch_gemv(a, as_stream(stream))
                                                       : launch_gemm_i8(a, as_stream(stream));
  return hip_status(e);
}

fairy2i_status fairy2i_host_exact_mean_f32(const double* values, int64_t n_values, float* out) {
  if (!out || (n_values > 0 && !values)) return FAIRY2I_ERR_NULL;
  if (n_values < 0 || n_values > FAIRY2I_MAX_QUANTIZE_ENTRIES) return FAIRY2I_ERR_SHAPE;
  if (n_values == 0) {
    *out = 0.0f;
    return FAIRY2I_OK;
  }
  std::vector<uint64_t> limbs(SA_LIMBS, 0);
  for (int64_t i = 0; i < n_values; ++i) {
    double v = values[i] < 0 ? -values[i] : values[i];
    if (v == 0.0) continue;
    int limb;
    uint32_t lo, mid, hi;
    sa_split(v, &limb, &lo, &mid, &hi);
    limbs[limb] += lo;
    limbs[limb + 1] += mid;
    limbs[limb + 2] += hi;
  }
  *out = sa_mean_to_f32(limbs.data(), (uint64_t)n_values);
  return FAIRY2I_OK;
}

}  // extern "C"
