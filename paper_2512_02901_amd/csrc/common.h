// Internal declarations shared by the kernels and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fairy2i.h"

namespace fairy2i {

// ---------------------------------------------------------------- to_wl ---
hipError_t launch_to_widely_linear(const float* A, int64_t N, int64_t K, float2* U, float2* W,
                                   hipStream_t stream);

// ------------------------------------------------------------- quantize ---
// Workspace layout of the quantiser: one partial superaccumulator per block.
constexpr int kQzThreads = 256;
constexpr int kQzMaxBlocks = 1024;
size_t quantize_workspace_bytes(int64_t N, int64_t K);
hipError_t launch_quantize_grouped(const float2* M, int64_t N, int64_t K, int T, int64_t G, uint8_t* codes,
                                   float* scales, hipStream_t stream);
hipError_t launch_quantize(const float2* M, int64_t N, int64_t K, int T, uint8_t* codes,
                           float* scales, void* workspace, hipStream_t stream);

// --------------------------------------------------------------- repack ---
size_t repack_tiled_bytes(int64_t N, int64_t K, int T);
hipError_t launch_repack_tiled(const uint8_t* codes, int64_t N, int64_t K, int T, uint8_t* tiled,
                               hipStream_t stream);
hipError_t launch_repack_fp4(const uint8_t* codes, int64_t N, int64_t K, int T, uint8_t* out,
                             hipStream_t stream);

// ----------------------------------------------------------- act quant ---
hipError_t launch_quantize_act_int8(const void* x, int dtype, int64_t B, int64_t K, int8_t* q,
                                    float* x_scale, hipStream_t stream);

// ------------------------------------------------------- wl products ---
struct WlArgs {
  const uint8_t* codes[2];   // U, W
  const float* scales[2];    // U, W ([T][2]); unused when exporting accumulators
  int T;
  int64_t N, K, B;
  const void* x;             // B*K*2 of dtype
  const float* x_scale;      // int8 only
  int dtype;
  float2* y;                 // [B][N] (epilogue mode)
  int32_t* acc;              // [2][T][2][B][N][2] (export mode), else null
};

hipError_t launch_gemv(const WlArgs& a, hipStream_t stream);       // B <= 16
// int8, any B.  With a workspace of gemm_workspace_bytes (> 0 only when
// K % 64 == 0 and sizes fit 32-bit offsets) the pipelined kernel runs, else
// the direct one.
size_t gemm_workspace_bytes(int64_t N, int64_t K, int64_t B);
hipError_t launch_gemm_i8(const WlArgs& a, void* workspace, hipStream_t stream);

}  // namespace fairy2i
