// Decode product for 1..16 tokens (Sec. 3.4, Algorithm 1, with the
// dequantisation of Eq. ifairy-dequant and the W conj(x) term).
//
// Multiplication-free accumulation: for each matrix M in {U, W}, stage t and
// axis a in {re, im} the kernel keeps one complex accumulator
//     A[M][t][a] = sum over codes k with (k & 1) == a of  (-1)^(k >> 1) x_j
// i.e. each 2-bit code costs one signed complex add of x_j into the
// accumulator its axis bit selects.  Both U and W accumulate x itself; the
// multiplication by i, the conjugation of the W term and the axis scales are
// applied once per output in the epilogue:
//     y = sum_t  s^U_re A[U][t][re] + i s^U_im A[U][t][im]
//              + s^W_re conj(A[W][t][re]) + i s^W_im conj(A[W][t][im]).
// Accumulation is float32 for float activations and exact int32 for int8.
//
// Layout: one wave per output row, four rows per block.  Lane l owns the
// 32-bit code word (16 codes) l of every 1024-code chunk of the row, for each
// of the 2T code planes; the chunk of activations is staged in LDS (padded to
// spread banks).  Partial sums are reduced across the wave with shuffles in a
// fixed order, so the result is bitwise reproducible.
#include "common.h"

namespace fairy2i {

namespace {

constexpr int kChunk = 1024;               // codes per LDS chunk
constexpr int kPad = kChunk + kChunk / 16;  // one float2 of padding every 16

__device__ inline int lds_index(int n) { return n + (n >> 4); }

template <int DT>
struct ActTraits;
template <>
struct ActTraits<FAIRY2I_ACT_F32> {
  using acc_t = float;
  __device__ static inline void load(const void* x, int64_t i, acc_t& re, acc_t& im) {
    const float2 v = static_cast<const float2*>(x)[i];
    re = v.x;
    im = v.y;
  }
};
template <>
struct ActTraits<FAIRY2I_ACT_BF16> {
  using acc_t = float;
  __device__ static inline void load(const void* x, int64_t i, acc_t& re, acc_t& im) {
    const uint32_t v = static_cast<const uint32_t*>(x)[i];
    re = __uint_as_float(v << 16);
    im = __uint_as_float(v & 0xFFFF0000u);
  }
};
template <>
struct ActTraits<FAIRY2I_ACT_I8> {
  using acc_t = int;
  __device__ static inline void load(const void* x, int64_t i, acc_t& re, acc_t& im) {
    const uint16_t v = static_cast<const uint16_t*>(x)[i];
    re = (int)(int8_t)(v & 0xFF);
    im = (int)(int8_t)(v >> 8);
  }
};

// 16 codes starting at code j0 of a row that has K codes, packed 4 per byte.
// Codes at or beyond K read as 0 (their activations are zero).
__device__ inline uint32_t load_code_word(const uint8_t* row, int64_t K, int64_t j0, bool aligned) {
  if (aligned) return *reinterpret_cast<const uint32_t*>(row + j0 / 4);
  uint32_t w = 0;
  for (int b = 0; b < 4; ++b)
    if (j0 + 4 * b < K) w |= (uint32_t)row[j0 / 4 + b] << (8 * b);
  return w;
}

template <typename A>
__device__ inline A wave_sum(A v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

template <int DT, int T, int TB, bool EXPORT>
__global__ __launch_bounds__(256) void gemv_valu_kernel(WlArgs a, bool aligned) {
  using Tr = ActTraits<DT>;
  using acc_t = typename Tr::acc_t;
  __shared__ acc_t xs[TB][kPad][2];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * 4 + wave;
  const bool row_ok = row < a.N;
  const int64_t b0 = (int64_t)blockIdx.y * TB;
  const int64_t K = a.K;
  const int64_t plane = a.N * K / 4;  // bytes per stage plane

  acc_t acc[2][T][2][TB][2];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int ax = 0; ax < 2; ++ax)
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) acc[m][t][ax][tb][0] = acc[m][t][ax][tb][1] = 0;

  for (int64_t c0 = 0; c0 < K; c0 += kChunk) {
    __syncthreads();
    for (int n = threadIdx.x; n < TB * kChunk; n += blockDim.x) {
      const int tb = n / kChunk, jj = n - tb * kChunk;
      const int64_t b = b0 + tb, j = c0 + jj;
      acc_t re = 0, im = 0;
      if (b < a.B && j < K) Tr::load(a.x, b * K + j, re, im);
      xs[tb][lds_index(jj)][0] = re;
      xs[tb][lds_index(jj)][1] = im;
    }
    __syncthreads();
    const int64_t j0 = c0 + 16 * lane;
    if (row_ok && j0 < K) {
#pragma unroll
      for (int m = 0; m < 2; ++m) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const uint8_t* rowp = a.codes[m] + t * plane + row * (K / 4);
          const uint32_t w = load_code_word(rowp, K, j0, aligned);
#pragma unroll
          for (int cc = 0; cc < 16; ++cc) {
            const uint32_t k = (w >> (2 * cc)) & 3u;
            const int li = lds_index(16 * lane + cc);
#pragma unroll
            for (int tb = 0; tb < TB; ++tb) {
              acc_t re = xs[tb][li][0], im = xs[tb][li][1];
              if (k & 2u) {
                re = -re;
                im = -im;
              }
              if (k & 1u) {
                acc[m][t][1][tb][0] += re;
                acc[m][t][1][tb][1] += im;
              } else {
                acc[m][t][0][tb][0] += re;
                acc[m][t][0][tb][1] += im;
              }
            }
          }
        }
      }
    }
  }

#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int ax = 0; ax < 2; ++ax)
#pragma unroll
        for (int tb = 0; tb < TB; ++tb) {
          acc[m][t][ax][tb][0] = wave_sum(acc[m][t][ax][tb][0]);
          acc[m][t][ax][tb][1] = wave_sum(acc[m][t][ax][tb][1]);
        }
  if (!row_ok || lane != 0) return;

#pragma unroll
  for (int tb = 0; tb < TB; ++tb) {
    const int64_t b = b0 + tb;
    if (b >= a.B) break;
    if constexpr (EXPORT) {
      // acc[M][t][p][b][i][c]
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
          for (int ax = 0; ax < 2; ++ax) {
            int32_t* dst = a.acc + ((((int64_t)(m * T + t) * 2 + ax) * a.B + b) * a.N + row) * 2;
            dst[0] = (int32_t)acc[m][t][ax][tb][0];
            dst[1] = (int32_t)acc[m][t][ax][tb][1];
          }
    } else {
      float yr = 0.0f, yi = 0.0f;
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const float su_re = a.scales[0][2 * t], su_im = a.scales[0][2 * t + 1];
        const float sw_re = a.scales[1][2 * t], sw_im = a.scales[1][2 * t + 1];
        const float ur0 = (float)acc[0][t][0][tb][0], ui0 = (float)acc[0][t][0][tb][1];
        const float ur1 = (float)acc[0][t][1][tb][0], ui1 = (float)acc[0][t][1][tb][1];
        const float wr0 = (float)acc[1][t][0][tb][0], wi0 = (float)acc[1][t][0][tb][1];
        const float wr1 = (float)acc[1][t][1][tb][0], wi1 = (float)acc[1][t][1][tb][1];
        yr += su_re * ur0 - su_im * ui1;
        yi += su_re * ui0 + su_im * ur1;
        yr += sw_re * wr0 + sw_im * wi1;
        yi += -sw_re * wi0 + sw_im * wr1;
      }
      if constexpr (DT == FAIRY2I_ACT_I8) {
        const float f = a.x_scale[b];
        yr *= f;
        yi *= f;
      }
      a.y[b * a.N + row] = make_float2(yr, yi);
    }
  }
}

template <int DT, int T, int TB, bool EXPORT>
hipError_t launch_tb(const WlArgs& a, hipStream_t s) {
  const bool aligned = (a.K % 16) == 0;
  dim3 grid((unsigned)((a.N + 3) / 4), (unsigned)((a.B + TB - 1) / TB));
  hipLaunchKernelGGL((gemv_valu_kernel<DT, T, TB, EXPORT>), grid, dim3(256), 0, s, a, aligned);
  return hipGetLastError();
}

template <int DT, int T, bool EXPORT>
hipError_t launch_t(const WlArgs& a, hipStream_t s) {
  if (a.B == 1) return launch_tb<DT, T, 1, EXPORT>(a, s);
  if (a.B == 2) return launch_tb<DT, T, 2, EXPORT>(a, s);
  return launch_tb<DT, T, 4, EXPORT>(a, s);
}

template <int DT, bool EXPORT>
hipError_t launch_dt(const WlArgs& a, hipStream_t s) {
  switch (a.T) {
    case 1: return launch_t<DT, 1, EXPORT>(a, s);
    case 2: return launch_t<DT, 2, EXPORT>(a, s);
    case 3: return launch_t<DT, 3, EXPORT>(a, s);
    default: return launch_t<DT, 4, EXPORT>(a, s);
  }
}

}  // namespace

hipError_t launch_gemv(const WlArgs& a, hipStream_t s) {
  if (a.acc) return launch_dt<FAIRY2I_ACT_I8, true>(a, s);
  switch (a.dtype) {
    case FAIRY2I_ACT_F32: return launch_dt<FAIRY2I_ACT_F32, false>(a, s);
    case FAIRY2I_ACT_BF16: return launch_dt<FAIRY2I_ACT_BF16, false>(a, s);
    default: return launch_dt<FAIRY2I_ACT_I8, false>(a, s);
  }
}

}  // namespace fairy2i
