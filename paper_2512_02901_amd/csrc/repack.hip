// D3 packed codes -> the tiled decode layouts: tiled (a byte permutation;
// the code values and their packing into bytes are unchanged) and fp4 tiled
// (the same tiles, code bits rearranged for the fp8 x fp4 matrix cores).
//
// Tile (row block rb, 256-code step s, stage t) is 1024 bytes at offset
// ((rb * nk4 + s) * T + t) * 1024; its byte 16 * lane + e (lane = 16 g + r)
// is D3 byte 64 s + 16 g + e of row 16 rb + r.  One thread writes one
// 16-byte chunk (one lane's share of a tile); rows past N and bytes past the
// row's K/4 are written as zeros.

#include "common.h"

namespace fairy2i {
namespace {

__global__ __launch_bounds__(256) void repack_tiled_kernel(const uint8_t* __restrict__ codes, int64_t N,
                                                           int64_t K, int T, int64_t nk4, uint4* __restrict__ out,
                                                           int64_t nchunks, bool vec) {
  const int64_t rowbytes = K / 4;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < nchunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int lane = (int)(c & 63);
    int64_t r = c >> 6;
    const int t = (int)(r % T);
    r /= T;
    const int64_t s = r % nk4;
    const int64_t rb = r / nk4;
    const int64_t row = rb * 16 + (lane & 15);
    const int64_t b0 = s * 64 + 16 * (lane >> 4);
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (row < N && b0 < rowbytes) {
      const uint8_t* src = codes + ((int64_t)t * N + row) * rowbytes + b0;
      if (vec) {
        v = *reinterpret_cast<const uint4*>(src);  // rowbytes % 16 == 0: the whole run is in the row
      } else {
        uint32_t w[4] = {0u, 0u, 0u, 0u};
        for (int e = 0; e < 16 && b0 + e < rowbytes; ++e) w[e >> 2] |= (uint32_t)src[e] << (8 * (e & 3));
        v = make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
    out[c] = v;
  }
}

// Fp4 tiled layout: the tiles of the tiled layout, with the 64 codes of a
// lane's 16 bytes rearranged for the fp8 x fp4 decode.  Lane (g, r) of tile
// (rb, s, t) holds codes 256 s + 128 kb + 32 g + n (kb < 2, n < 32) of row
// 16 rb + r; with n = 16 h + 8 a + m, code n sits in word 2 kb + h, nibble m,
// at bits (3, 1) = (q, p) for a = 0 and bits (2, 0) = (q, p) for a = 1,
// where p, q are bits 0 and 1 of the code.  Padding codes are 0.
__global__ __launch_bounds__(256) void repack_fp4_kernel(const uint8_t* __restrict__ codes, int64_t N, int64_t K,
                                                         int T, int64_t nk4, uint4* __restrict__ out,
                                                         int64_t nchunks) {
  const int64_t rowbytes = K / 4;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < nchunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int lane = (int)(c & 63);
    int64_t r = c >> 6;
    const int t = (int)(r % T);
    r /= T;
    const int64_t s = r % nk4;
    const int64_t rb = r / nk4;
    const int64_t row = rb * 16 + (lane & 15);
    const int g = lane >> 4;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    if (row < N) {
      const uint8_t* src = codes + ((int64_t)t * N + row) * rowbytes;
      for (int kb = 0; kb < 2; ++kb) {
        const int64_t b0 = s * 64 + kb * 32 + g * 8;  // D3 bytes of codes 256 s + 128 kb + 32 g + n
        for (int n = 0; n < 32; ++n) {
          const int64_t byte = b0 + (n >> 2);
          if (byte >= rowbytes) break;
          const uint32_t code = (src[byte] >> (2 * (n & 3))) & 3u;
          const uint32_t p = code & 1u, q = code >> 1;
          const int h = n >> 4, a = (n >> 3) & 1, m = n & 7;
          const uint32_t nib = a == 0 ? (q << 3) | (p << 1) : (q << 2) | p;
          w[2 * kb + h] |= nib << (4 * m);
        }
      }
    }
    out[c] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

}  // namespace

hipError_t launch_repack_fp4(const uint8_t* codes, int64_t N, int64_t K, int T, uint8_t* out,
                             hipStream_t stream) {
  const int64_t nk4 = (K + 255) / 256;
  const int64_t nchunks = (int64_t)repack_tiled_bytes(N, K, T) / 16;
  int64_t blocks = (nchunks + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(repack_fp4_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, codes, N, K, T, nk4,
                     reinterpret_cast<uint4*>(out), nchunks);
  return hipGetLastError();
}

size_t repack_tiled_bytes(int64_t N, int64_t K, int T) {
  return (size_t)T * (size_t)((N + 15) / 16) * (size_t)((K + 255) / 256) * 1024;
}

hipError_t launch_repack_tiled(const uint8_t* codes, int64_t N, int64_t K, int T, uint8_t* tiled,
                               hipStream_t stream) {
  const int64_t nk4 = (K + 255) / 256;
  const int64_t nchunks = (int64_t)repack_tiled_bytes(N, K, T) / 16;
  const bool vec = (K / 4) % 16 == 0 && (reinterpret_cast<uintptr_t>(codes) & 15) == 0;
  int64_t blocks = (nchunks + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(repack_tiled_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, codes, N, K, T, nk4,
                     reinterpret_cast<uint4*>(tiled), nchunks, vec);
  return hipGetLastError();
}

}  // namespace fairy2i
