// Real form of a widely-linear layer for training (Sec. 3.1, Eq. UW-from-R
// read backwards, with Eq. realify-ops): y = U x + W conj(x) is one real
// linear map of the stacked (Re, Im) pairs, whose 2 x 2 block for output n
// and input k is
//     [ Re U + Re W    Im W - Im U ]
//     [ Im U + Im W    Re U - Re W ]
// (R11 = Re U + Re W, R12 = Im W - Im U, R21 = Im U + Im W, R22 = Re U - Re W
// of the half-split real matrix).  With R stored interleaved (row 2n + a,
// column 2k + b for the (a, b) entry of that block) and tokens stored as
// (re, im) pairs, the three products of a training step are plain real
// GEMMs of the same data in place:
//     Y   = X R^T        (M x 2N  =  M x 2K  .  2K x 2N)
//     G_X = G_Y R        (the gradient through the real map)
//     G_R = G_Y^T X      (2N x 2K)
// and G_U = G_Y^T conj(X), G_W = G_Y^T X are read off G_R's blocks:
//     Re G_U = G_R[2n][2k] + G_R[2n+1][2k+1],  Im G_U = G_R[2n+1][2k] - G_R[2n][2k+1],
//     Re G_W = G_R[2n][2k] - G_R[2n+1][2k+1],  Im G_W = G_R[2n][2k+1] + G_R[2n+1][2k].
// Against Gauss's three complex products per segment (six real products of
// M x N x K for the two segments) this is four real products' work, and the
// operands need no planes.
#include "common.h"

namespace fairy2i {

namespace {

__device__ inline uint16_t bf16_rne_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// A double rounded once to bf16 (nearest even).  Rounding to float32 first
// and then to bf16 goes wrong only where the float32 value is a bf16 tie
// that the double is not on (every bf16 tie is a float32 value, so
// elsewhere the float32 value lies on the same side of every tie as the
// double); there the sign of the float32 rounding's remainder decides.
// (Selects, no branches: at a float32 tie f is not zero, so a nonzero
// remainder rounds away from zero exactly when it has f's sign.)
__device__ inline uint16_t bf16_from_double(double v) {
  const float f = (float)v;  // nearest float32
  const double r = v - (double)f;
  const uint32_t u = __float_as_uint(f);
  const uint32_t low = u & 0xFFFFu;
  const uint32_t hi = u >> 16;
  const uint32_t away = r != 0.0 ? (uint32_t)((r > 0.0) == (f > 0.0f)) : (hi & 1u);
  return (uint16_t)(hi + ((uint32_t)(low > 0x8000u) | ((uint32_t)(low == 0x8000u) & away)));
}

__device__ inline float2 load_c(const void* p, int32_t dtype, int64_t i) {
  if (dtype == FAIRY2I_ACT_BF16) {
    const uint32_t w = static_cast<const uint32_t*>(p)[i];
    return make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
  }
  return static_cast<const float2*>(p)[i];
}

// One thread per (n, k): the block's four entries as two 32-bit words, one
// in row 2n and one in row 2n + 1.
__global__ __launch_bounds__(256) void realify_kernel(const void* __restrict__ U, const void* __restrict__ W,
                                                      int32_t dtype, int64_t N, int64_t K,
                                                      uint32_t* __restrict__ R) {
  const int64_t total = N * K;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    // N K <= 2^30 (checked by the host): 32-bit division
    const int64_t n = (int64_t)((uint32_t)i / (uint32_t)K), k = i - n * K;
    const float2 u = load_c(U, dtype, i), w = load_c(W, dtype, i);
    const double ur = u.x, ui = u.y, wr = w.x, wi = w.y;
    const uint32_t top = (uint32_t)bf16_from_double(ur + wr) | ((uint32_t)bf16_from_double(wi - ui) << 16);
    const uint32_t bot = (uint32_t)bf16_from_double(ui + wi) | ((uint32_t)bf16_from_double(ur - wr) << 16);
    R[(2 * n) * K + k] = top;      // row 2n: columns 2k, 2k + 1 (K words per row)
    R[(2 * n + 1) * K + k] = bot;  // row 2n + 1
  }
}

// One thread per (n, k): G_U and G_W from the block of G_R (float32 sums).
__global__ __launch_bounds__(256) void unrealify_grad_kernel(const float2* __restrict__ GR, int64_t N, int64_t K,
                                                             float2* __restrict__ GU, float2* __restrict__ GW) {
  const int64_t total = N * K;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t n = (int64_t)((uint32_t)i / (uint32_t)K), k = i - n * K;  // N K <= 2^30
    const float2 t = GR[(2 * n) * K + k];      // (G_R[2n][2k], G_R[2n][2k+1])
    const float2 b = GR[(2 * n + 1) * K + k];  // (G_R[2n+1][2k], G_R[2n+1][2k+1])
    GU[i] = make_float2(t.x + b.y, b.x - t.y);
    GW[i] = make_float2(t.x - b.y, t.y + b.x);
  }
}

// R straight from the codes (Eq. ifairy-dequant, Eq. res-sum): one thread
// per packed byte, i.e. four entries (n, 4 j .. 4 j + 3) of U and of W, each
// summed over the stages in increasing order in double (as the fake-quant
// dequantisation does), their block entries formed in double and rounded
// once to bf16; a 16-byte store per row of the block pair.  A stage adds
// s c with c in {1, 0, -1} as one fused multiply-add: the same rounding as
// adding or subtracting s, or nothing (a sum never holds -0, and the scales
// are not negative), without a branch on the code.
__global__ __launch_bounds__(256) void realify_codes_kernel(const uint8_t* __restrict__ cu,
                                                            const float* __restrict__ su,
                                                            const uint8_t* __restrict__ cw,
                                                            const float* __restrict__ sw, int T, int64_t N,
                                                            int64_t K, uint4* __restrict__ R) {
  const int64_t nbytes = N * K / 4, kb = K / 4;
  for (int64_t bi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; bi < nbytes;
       bi += (int64_t)gridDim.x * blockDim.x) {
    double ur[4] = {0.0, 0.0, 0.0, 0.0}, ui[4] = {0.0, 0.0, 0.0, 0.0};
    double wr[4] = {0.0, 0.0, 0.0, 0.0}, wi[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int t = 0; t < FAIRY2I_MAX_STAGES; ++t) {
      if (t >= T) break;
      const uint32_t bu = cu[(int64_t)t * nbytes + bi], bw = cw[(int64_t)t * nbytes + bi];
      const double sur = (double)su[2 * t], sui = (double)su[2 * t + 1];
      const double swr = (double)sw[2 * t], swi = (double)sw[2 * t + 1];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ku = (int)((bu >> (2 * e)) & 3u), kw = (int)((bw >> (2 * e)) & 3u);
        // i^k: 0 -> +1, 1 -> +i, 2 -> -1, 3 -> -i: real part 1 - k for even k, imaginary part 2 - k for odd k
        const int cur = (1 - ku) & ((ku & 1) - 1), cui = (2 - ku) & -(ku & 1);
        const int cwr = (1 - kw) & ((kw & 1) - 1), cwi = (2 - kw) & -(kw & 1);
        ur[e] = fma(sur, (double)cur, ur[e]);
        ui[e] = fma(sui, (double)cui, ui[e]);
        wr[e] = fma(swr, (double)cwr, wr[e]);
        wi[e] = fma(swi, (double)cwi, wi[e]);
      }
    }
    uint32_t top[4], bot[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      top[e] = (uint32_t)bf16_from_double(ur[e] + wr[e]) | ((uint32_t)bf16_from_double(wi[e] - ui[e]) << 16);
      bot[e] = (uint32_t)bf16_from_double(ui[e] + wi[e]) | ((uint32_t)bf16_from_double(ur[e] - wr[e]) << 16);
    }
    const int64_t n = (int64_t)((uint32_t)bi / (uint32_t)kb), j = bi - n * kb;  // N K / 4 <= 2^28
    R[(2 * n) * kb + j] = make_uint4(top[0], top[1], top[2], top[3]);  // row 2n: K words, K / 4 uint4
    R[(2 * n + 1) * kb + j] = make_uint4(bot[0], bot[1], bot[2], bot[3]);
  }
}

__global__ __launch_bounds__(256) void f32_to_bf16_kernel(const float* __restrict__ in, int64_t n,
                                                          uint16_t* __restrict__ out) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    out[i] = bf16_rne_bits(in[i]);
}

inline unsigned grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b > 65536) b = 65536;
  return (unsigned)(b < 1 ? 1 : b);
}

}  // namespace

}  // namespace fairy2i

using namespace fairy2i;

extern "C" {

fairy2i_status fairy2i_wl_realify(const void* U, const void* W, int32_t dtype, int64_t N, int64_t K, void* R,
                                  void* stream) {
  if (!U || !W || !R) return FAIRY2I_ERR_NULL;
  if (dtype != FAIRY2I_ACT_F32 && dtype != FAIRY2I_ACT_BF16) return FAIRY2I_ERR_DTYPE;
  if (N <= 0 || K <= 0 || N > ((int64_t)1 << 30) / K) return FAIRY2I_ERR_SHAPE;
  hipLaunchKernelGGL(realify_kernel, dim3(grid_for(N * K)), dim3(256), 0, static_cast<hipStream_t>(stream), U, W,
                     dtype, N, K, static_cast<uint32_t*>(R));
  return hipGetLastError() == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP;
}

fairy2i_status fairy2i_wl_realify_codes(const uint8_t* codes_U, const float* scales_U, const uint8_t* codes_W,
                                        const float* scales_W, int32_t T, int64_t N, int64_t K, void* R,
                                        void* stream) {
  if (!codes_U || !scales_U || !codes_W || !scales_W || !R) return FAIRY2I_ERR_NULL;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (N <= 0 || K <= 0 || K % 4 != 0 || N > ((int64_t)1 << 30) / K) return FAIRY2I_ERR_SHAPE;
  if (reinterpret_cast<uintptr_t>(R) & 15) return FAIRY2I_ERR_SHAPE;
  hipLaunchKernelGGL(realify_codes_kernel, dim3(grid_for(N * K / 4)), dim3(256), 0, static_cast<hipStream_t>(stream),
                     codes_U, scales_U, codes_W, scales_W, T, N, K, static_cast<uint4*>(R));
  return hipGetLastError() == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP;
}

fairy2i_status fairy2i_wl_unrealify_grad(const float* G_R, int64_t N, int64_t K, float* G_U, float* G_W,
                                         void* stream) {
  if (!G_R || !G_U || !G_W) return FAIRY2I_ERR_NULL;
  if (N <= 0 || K <= 0 || N > ((int64_t)1 << 30) / K) return FAIRY2I_ERR_SHAPE;
  hipLaunchKernelGGL(unrealify_grad_kernel, dim3(grid_for(N * K)), dim3(256), 0, static_cast<hipStream_t>(stream),
                     reinterpret_cast<const float2*>(G_R), N, K, reinterpret_cast<float2*>(G_U),
                     reinterpret_cast<float2*>(G_W));
  return hipGetLastError() == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP;
}

fairy2i_status fairy2i_f32_to_bf16(const float* in, int64_t n, void* out, void* stream) {
  if (!in || !out) return FAIRY2I_ERR_NULL;
  if (n <= 0) return FAIRY2I_ERR_SHAPE;
  hipLaunchKernelGGL(f32_to_bf16_kernel, dim3(grid_for(n)), dim3(256), 0, static_cast<hipStream_t>(stream), in, n,
                     static_cast<uint16_t*>(out));
  return hipGetLastError() == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP;
}

}  // extern "C"
