// Decode (1..16 token) product on the int8 matrix cores: internal layer
// descriptors shared by the C-ABI layer and decode.hip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fairy2i {

constexpr int kModeBf16 = 0;  // bf16 activations as 3 base-256 digits of a 23-bit fixed point
constexpr int kModeI8 = 1;    // int8 activations with a per-token factor
constexpr int kDecKc4 = 2;    // 256-code steps per work item (512 codes)
constexpr int kDecMaxBlocks = 8192;

// One layer of a decode call.  Workspace pointers (xf, xs, part) are carved
// out of the caller's workspace by the host code.
struct DecLayer {
  const uint8_t* codes[2];   // U, W: [T][N][K/4]
  const float* scales[2];    // U, W: [T][2]
  const void* x;             // [B][K][2] bf16 or int8
  const float* x_scale_in;   // int8: [B] dequantisation factors
  float2* y;                 // [B][N]
  int32_t* acc;              // accumulator export [2][T][2][B][N][2], else null
  int8_t* xf;                // activation operand [ntile][nk4][4][64][16]
  float* xs;                 // per-token output factor [B]
  float2* part;              // split-K partials [nkc][B][N] (nkc > 1)
  int32_t N, K;
  int32_t nrb, nk4, nkc, pad_;
  int64_t item0;             // index of this layer's first work item
};

struct DecHeader {
  int32_t n_layers, T, mode, B, ntile, pad_;
  int64_t total_items;
};

// Tiles of 16 activation columns processed per pass over a work item.
int dec_tiles_per_group(int T, int ntile);

// Fill the geometry fields of `l` (N, K set) and return its workspace bytes.
// With `ws` non-null, also carve xf, xs, part out of it.
size_t dec_layer_setup(DecLayer& l, int T, int mode, int B, char* ws);

hipError_t launch_decode(const DecHeader& h, const DecLayer& inl, const DecLayer* tab,
                         int any_split, int64_t max_BN, bool export_acc, int64_t acc_elems,
                         int32_t* acc, hipStream_t s, hipEvent_t const* events = nullptr);

}  // namespace fairy2i
