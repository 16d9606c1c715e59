// Prefill product with int8 activations on the int8 matrix cores (gfx950
// v_mfma_i32_16x16x64_i8).
//
// Each code i^k is the 2x2 real block b_re I + b_im J of Eq. (realify-ops)
// with (b_re, b_im) in {(1,0), (0,1), (-1,0), (0,-1)}.  Because the two
// axis scales differ, the two ternary planes B_re, B_im in {-1,0,+1}^{N x K}
// are contracted separately:
//     P[M][t][p] = B^{M,t}_p  .  [q_re | q_im]      (exact int32)
// i.e. one dense int8 GEMM of (4T N) x K x (2 tokens), whose int32 results
// are combined per output in registers (scales, the factor i, the
// conjugation of the W term, the sum over stages, the token's dequantisation
// factor), never written out.
//
// Tile: a block of 4 waves covers 32 output rows x 2*TOKW tokens; wave w
// owns rows 16*(w&1) .. +16 and tokens TOKW*(w>>1) .. +TOKW, for all 4T
// (M, t, plane) groups, so every accumulator an output needs sits in the
// same lane.  Per 64-code step:
//   * activations of the block's tokens are staged in LDS, split into re and
//     im planes, with each 16-code group stored in the order the expanded
//     codes use (byte 4c+b of a group holds code c + 4b);
//   * each wave loads, per (M, t), one 32-bit code word (16 codes) per lane
//     straight from global memory and expands it in registers with v_perm
//     byte tables into the b_re and b_im int8 planes (the selector byte for
//     code c + 4b is (word >> 2c) & 3 in byte b);
//   * 2 MFMAs per (M, t) and B-fragment.
#include "common.h"

namespace fairy2i {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr uint32_t kTableRe = 0x00FF0001u;  // code 0 -> +1, 1 -> 0, 2 -> -1, 3 -> 0
constexpr uint32_t kTableIm = 0xFF000100u;  // code 0 -> 0, 1 -> +1, 2 -> 0, 3 -> -1
constexpr int kRowPad = 80;                 // bytes per LDS token row (64 + 16 pad)

__device__ inline uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// Expand 16 codes into the int8 b_re and b_im planes of one MFMA A fragment.
__device__ inline void expand_codes(uint32_t w, v4i& are, v4i& aim) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const uint32_t sel = (w >> (2 * c)) & 0x03030303u;
    are[c] = (int)perm(0u, kTableRe, sel);
    aim[c] = (int)perm(0u, kTableIm, sel);
  }
}

// 32 bytes = 16 codes x (re, im) interleaved -> 16 re bytes and 16 im bytes,
// each in the expanded-code order (byte 4d+b holds code d + 4b).
__device__ inline void split_group(const uint32_t I[8], uint32_t re[4], uint32_t im[4]) {
  // bytes: I[n] holds codes 2n (b0 re, b1 im) and 2n+1 (b2 re, b3 im)
  const uint32_t r02 = perm(I[2], I[0], 0x06020400u), r46 = perm(I[6], I[4], 0x06020400u);
  const uint32_t r13 = perm(I[3], I[1], 0x06020400u), r57 = perm(I[7], I[5], 0x06020400u);
  const uint32_t i02 = perm(I[2], I[0], 0x07030501u), i46 = perm(I[6], I[4], 0x07030501u);
  const uint32_t i13 = perm(I[3], I[1], 0x07030501u), i57 = perm(I[7], I[5], 0x07030501u);
  re[0] = perm(r46, r02, 0x05040100u);
  re[1] = perm(r46, r02, 0x07060302u);
  re[2] = perm(r57, r13, 0x05040100u);
  re[3] = perm(r57, r13, 0x07060302u);
  im[0] = perm(i46, i02, 0x05040100u);
  im[1] = perm(i46, i02, 0x07060302u);
  im[2] = perm(i57, i13, 0x05040100u);
  im[3] = perm(i57, i13, 0x07060302u);
}

__device__ inline uint32_t load_code_word(const uint8_t* row, int64_t K, int64_t j0, bool aligned) {
  if (j0 >= K) return 0u;
  if (aligned) return *reinterpret_cast<const uint32_t*>(row + j0 / 4);
  uint32_t w = 0;
  for (int b = 0; b < 4; ++b)
    if (j0 + 4 * b < K) w |= (uint32_t)row[j0 / 4 + b] << (8 * b);
  return w;
}

template <int T, int TOKW, bool EXPORT>
__global__ __launch_bounds__(256) void gemm_i8_kernel(WlArgs a, bool aligned) {
  constexpr int NTG = TOKW / 16;    // 16-token groups per wave
  constexpr int TOKB = 2 * TOKW;    // tokens per block
  __shared__ __attribute__((aligned(16))) int8_t xs[2][TOKB][kRowPad];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int rh = wave & 1, th = wave >> 1;
  const int64_t K = a.K;
  const int64_t row0 = (int64_t)blockIdx.x * 32 + 16 * rh;
  const int64_t tok0 = (int64_t)blockIdx.y * TOKB;
  const int64_t plane = a.N * K / 4;

  // A-fragment row of this lane (clamped to a valid row; results for rows
  // >= N are never stored).
  int64_t arow = row0 + (lane & 15);
  if (arow >= a.N) arow = a.N - 1;
  const int g = lane >> 4;

  v4i acc[2][T][2][NTG][2];
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int t = 0; t < T; ++t)
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int tg = 0; tg < NTG; ++tg)
#pragma unroll
          for (int c = 0; c < 2; ++c) acc[m][t][p][tg][c] = v4i{0, 0, 0, 0};

  const int8_t* q = static_cast<const int8_t*>(a.x);

  for (int64_t k0 = 0; k0 < K; k0 += 64) {
    __syncthreads();
    // ---- stage activations: TOKB tokens x 4 groups of 16 codes ----
    for (int u = tid; u < TOKB * 4; u += 256) {
      const int tl = u >> 2, part = u & 3;
      const int64_t tok = tok0 + tl;
      const int64_t kk = k0 + 16 * part;
      uint32_t I[8];
      if (tok < a.B && kk + 16 <= K && aligned) {
        const uint4* src = reinterpret_cast<const uint4*>(q + (tok * K + kk) * 2);
        const uint4 v0 = src[0], v1 = src[1];
        I[0] = v0.x; I[1] = v0.y; I[2] = v0.z; I[3] = v0.w;
        I[4] = v1.x; I[5] = v1.y; I[6] = v1.z; I[7] = v1.w;
      } else {
        for (int n = 0; n < 8; ++n) I[n] = 0u;
        if (tok < a.B) {
          for (int e = 0; e < 32; ++e) {
            const int64_t j = kk + (e >> 1);
            if (j < K) I[e >> 2] |= (uint32_t)(uint8_t)q[(tok * K + kk) * 2 + e] << (8 * (e & 3));
          }
        }
      }
      uint32_t re[4], im[4];
      split_group(I, re, im);
      *reinterpret_cast<uint4*>(&xs[0][tl][16 * part]) = make_uint4(re[0], re[1], re[2], re[3]);
      *reinterpret_cast<uint4*>(&xs[1][tl][16 * part]) = make_uint4(im[0], im[1], im[2], im[3]);
    }
    __syncthreads();

    // ---- B fragments from LDS ----
    v4i bfrag[NTG][2];
#pragma unroll
    for (int tg = 0; tg < NTG; ++tg)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        bfrag[tg][c] = *reinterpret_cast<const v4i*>(&xs[c][TOKW * th + 16 * tg + (lane & 15)][16 * g]);

    // ---- A fragments from the codes, MFMAs ----
#pragma unroll
    for (int m = 0; m < 2; ++m) {
#pragma unroll
      for (int t = 0; t < T; ++t) {
        const uint8_t* rowp = a.codes[m] + t * plane + arow * (K / 4);
        const uint32_t w = load_code_word(rowp, K, k0 + 16 * g, aligned);
        v4i are, aim;
        expand_codes(w, are, aim);
#pragma unroll
        for (int tg = 0; tg < NTG; ++tg)
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            acc[m][t][0][tg][c] =
                __builtin_amdgcn_mfma_i32_16x16x64_i8(are, bfrag[tg][c], acc[m][t][0][tg][c], 0, 0, 0);
            acc[m][t][1][tg][c] =
                __builtin_amdgcn_mfma_i32_16x16x64_i8(aim, bfrag[tg][c], acc[m][t][1][tg][c], 0, 0, 0);
          }
      }
    }
  }

  // ---- epilogue: lane holds rows 4*(lane/16)+r, token column lane%16 ----
#pragma unroll
  for (int tg = 0; tg < NTG; ++tg) {
    const int64_t tok = tok0 + TOKW * th + 16 * tg + (lane & 15);
    if (tok >= a.B) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = row0 + 4 * (lane >> 4) + r;
      if (row >= a.N) continue;
      if constexpr (EXPORT) {
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
          for (int t = 0; t < T; ++t)
#pragma unroll
            for (int p = 0; p < 2; ++p) {
              int32_t* dst = a.acc + ((((int64_t)(m * T + t) * 2 + p) * a.B + tok) * a.N + row) * 2;
              dst[0] = acc[m][t][p][tg][0][r];
              dst[1] = acc[m][t][p][tg][1][r];
            }
      } else {
        float yr = 0.0f, yi = 0.0f;
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const float su_re = a.scales[0][2 * t], su_im = a.scales[0][2 * t + 1];
          const float sw_re = a.scales[1][2 * t], sw_im = a.scales[1][2 * t + 1];
          const float ur0 = (float)acc[0][t][0][tg][0][r], ui0 = (float)acc[0][t][0][tg][1][r];
          const float ur1 = (float)acc[0][t][1][tg][0][r], ui1 = (float)acc[0][t][1][tg][1][r];
          const float wr0 = (float)acc[1][t][0][tg][0][r], wi0 = (float)acc[1][t][0][tg][1][r];
          const float wr1 = (float)acc[1][t][1][tg][0][r], wi1 = (float)acc[1][t][1][tg][1][r];
          yr += su_re * ur0 - su_im * ui1;
          yi += su_re * ui0 + su_im * ur1;
          yr += sw_re * wr0 + sw_im * wi1;
          yi += -sw_re * wi0 + sw_im * wr1;
        }
        const float f = a.x_scale[tok];
        a.y[tok * a.N + row] = make_float2(yr * f, yi * f);
      }
    }
  }
}

// ------------------------------------------------------ pipelined GEMM ---
// Used when K % 64 == 0.  A prep pass writes the activations once in the
// exact MFMA operand layout
//     xp[16-token fragment f][64-code step s][component c][lane][16 bytes]
// (lane = 16 g + n: token 16 f + n, codes 64 s + 16 g .. +15 in the order the
// expanded codes use), so the GEMM moves operands with direct-to-LDS loads
// only.  A block of 4 waves covers 32 code rows x 64 tokens (wave w: rows
// 16 (w & 1) .. +16, fragments 2 (w >> 1) .. +2) and walks K in stages of 128
// codes, double-buffered in LDS: the loads of stage s+1 are in flight while
// stage s is multiplied.  Per stage and wave: one activation fragment (two
// steps x two components, 4 KB) and up to two 1 KB code tiles (32 rows x 32
// bytes of one (M, t) plane).

constexpr uint32_t kOobG = 0xFFFFFFF0u;  // buffer offset past every range: loads return 0
typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__global__ __launch_bounds__(256) void prefill_prep_kernel(const int8_t* __restrict__ q, int64_t B, int64_t K,
                                                          int64_t nks, uint4* __restrict__ xp, int64_t nchunks,
                                                          bool vec) {
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < nchunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int lane = (int)(c & 63);
    int64_t r = c >> 6;
    const int comp = (int)(r & 1);
    r >>= 1;
    const int64_t st = r % nks, f = r / nks;
    const int64_t tok = 16 * f + (lane & 15);
    const int64_t k0 = 64 * st + 16 * (lane >> 4);
    uint32_t out[4] = {0u, 0u, 0u, 0u};
    if (tok < B) {  // K % 64 == 0: the run k0 .. k0+15 is inside the row
      const int8_t* src = q + (tok * K + k0) * 2;
      int v[16];
      if (vec) {
        const uint4 w0 = reinterpret_cast<const uint4*>(src)[0], w1 = reinterpret_cast<const uint4*>(src)[1];
        const uint32_t wd[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          v[2 * i] = (int)(int8_t)(wd[i] >> (8 * comp));
          v[2 * i + 1] = (int)(int8_t)(wd[i] >> (16 + 8 * comp));
        }
      } else {
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] = src[2 * i + comp];
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int dd = e >> 2, bb = e & 3;  // byte 4dd+bb holds code dd + 4bb of the run
        out[dd] |= ((uint32_t)v[dd + 4 * bb] & 0xFFu) << (8 * bb);
      }
    }
    xp[c] = make_uint4(out[0], out[1], out[2], out[3]);
  }
}

template <int T, bool EXPORT>
__global__ __launch_bounds__(256, (T <= 3) ? 2 : 1) void gemm_i8_pipe_kernel(WlArgs a, const int8_t* __restrict__ xp) {
#if defined(__HIP_DEVICE_COMPILE__)  // LDS-DMA and buffer-descriptor code: device pass only
  constexpr int P = 2 * T;
  constexpr int CL = (P + 3) / 4;  // code tiles loaded per wave and stage
  __shared__ __attribute__((aligned(16))) uint8_t lx0[4][2][2][1024];  // [fragment][step][component]
  __shared__ __attribute__((aligned(16))) uint8_t lx1[4][2][2][1024];
  __shared__ __attribute__((aligned(16))) uint8_t lc0[P][1024];        // [plane][row (32) x 32 bytes]
  __shared__ __attribute__((aligned(16))) uint8_t lc1[P][1024];

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int rh = wave & 1, th = wave >> 1;
  const int64_t K = a.K;
  const int nks = (int)(K / 64);
  const int nst = (nks + 1) / 2;
  const int64_t row0 = (int64_t)blockIdx.x * 32;
  const int64_t f0 = (int64_t)blockIdx.y * 4;
  const int64_t nfrag = (a.B + 15) / 16;
  const uint32_t plane_bytes = (uint32_t)(a.N * K / 4);
  const __amdgpu_buffer_rsrc_t xr = rsrc(xp, (uint32_t)(nfrag * nks * 2048));

  // code tiles: lane l fetches row l/2, 16-byte half l%2 of the stage's 32 bytes
  const int64_t crow = row0 + (lane >> 1);
  const bool crow_ok = crow < a.N;
  const uint32_t cbase = crow_ok ? (uint32_t)(crow * (K / 4)) + 16u * (uint32_t)(lane & 1) : 0u;
  const int64_t xf = f0 + wave;  // the activation fragment this wave fetches
  const bool xf_ok = xf < nfrag;

  auto issue = [&](int st, uint8_t (*lx)[2][2][1024], uint8_t (*lc)[1024]) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int sidx = 2 * st + sub;
        const uint32_t off =
            (xf_ok && sidx < nks) ? (uint32_t)(((xf * nks + sidx) * 2 + c) * 1024) + (uint32_t)lane * 16u : kOobG;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_ptr_t)&lx[wave][sub][c][0], 16, off, 0, 0, 0);
      }
#pragma unroll
    for (int j = 0; j < CL; ++j) {
      const int p = (wave + 4 * j) % P;  // with P < 4j planes some waves repeat a tile (same bytes)
      const int m = p / T, t = p % T;
      const uint32_t half = (uint32_t)st * 32u + 16u * (uint32_t)(lane & 1);
      const uint32_t off = (crow_ok && half < (uint32_t)(K / 4)) ? cbase + (uint32_t)st * 32u : kOobG;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc(a.codes[m] + (int64_t)t * plane_bytes, plane_bytes),
                                               (lds_ptr_t)&lc[p][0], 16, off, 0, 0, 0);
    }
  };

  v4i acc[P][2][2][2];  // [plane (M, t)][axis][token fragment][component]
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int ax = 0; ax < 2; ++ax)
#pragma unroll
      for (int tg = 0; tg < 2; ++tg)
#pragma unroll
        for (int c = 0; c < 2; ++c) acc[p][ax][tg][c] = v4i{0, 0, 0, 0};

  const int arow = 16 * rh + (lane & 15);
  const int g = lane >> 4;
  auto compute = [&](int st, uint8_t (*lx)[2][2][1024], uint8_t (*lc)[1024]) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      if (2 * st + sub >= nks) break;
      v4i bq[2][2];
#pragma unroll
      for (int tg = 0; tg < 2; ++tg)
#pragma unroll
        for (int c = 0; c < 2; ++c) bq[tg][c] = *reinterpret_cast<const v4i*>(&lx[2 * th + tg][sub][c][lane * 16]);
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(&lc[p][arow * 32 + sub * 16 + 4 * g]);
        v4i are, aim;
        expand_codes(w, are, aim);
#pragma unroll
        for (int tg = 0; tg < 2; ++tg)
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            acc[p][0][tg][c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(are, bq[tg][c], acc[p][0][tg][c], 0, 0, 0);
            acc[p][1][tg][c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aim, bq[tg][c], acc[p][1][tg][c], 0, 0, 0);
          }
      }
    }
  };

  // stages alternate between the two buffers; the buffer index is a
  // compile-time choice so loads into one buffer never order reads of the other
  // One barrier per stage: after it, every wave has both received stage st
  // (each waited for its own loads) and finished stage st-1, whose buffer
  // the loads of stage st+1 then refill while stage st is multiplied.
  issue(0, lx0, lc0);
  for (int st = 0; st < nst; st += 2) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (st + 1 < nst) issue(st + 1, lx1, lc1);
    compute(st, lx0, lc0);
    if (st + 1 >= nst) break;
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (st + 2 < nst) issue(st + 2, lx0, lc0);
    compute(st + 1, lx1, lc1);
  }

  // ---- epilogue: lane holds rows 4*(lane/16)+r, token column lane%16 ----
#pragma unroll
  for (int tg = 0; tg < 2; ++tg) {
    const int64_t tok = 16 * (f0 + 2 * th + tg) + (lane & 15);
    if (tok >= a.B) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t row = row0 + 16 * rh + 4 * (lane >> 4) + r;
      if (row >= a.N) continue;
      if constexpr (EXPORT) {
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
          for (int ax = 0; ax < 2; ++ax) {
            int32_t* dst = a.acc + ((((int64_t)p * 2 + ax) * a.B + tok) * a.N + row) * 2;
            dst[0] = acc[p][ax][tg][0][r];
            dst[1] = acc[p][ax][tg][1][r];
          }
      } else {
        float yr = 0.0f, yi = 0.0f;
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const float su_re = a.scales[0][2 * t], su_im = a.scales[0][2 * t + 1];
          const float sw_re = a.scales[1][2 * t], sw_im = a.scales[1][2 * t + 1];
          const int pu = t, pw = T + t;
          const float ur0 = (float)acc[pu][0][tg][0][r], ui0 = (float)acc[pu][0][tg][1][r];
          const float ur1 = (float)acc[pu][1][tg][0][r], ui1 = (float)acc[pu][1][tg][1][r];
          const float wr0 = (float)acc[pw][0][tg][0][r], wi0 = (float)acc[pw][0][tg][1][r];
          const float wr1 = (float)acc[pw][1][tg][0][r], wi1 = (float)acc[pw][1][tg][1][r];
          yr += su_re * ur0 - su_im * ui1;
          yi += su_re * ui0 + su_im * ur1;
          yr += sw_re * wr0 + sw_im * wi1;
          yi += -sw_re * wi0 + sw_im * wr1;
        }
        const float f = a.x_scale[tok];
        a.y[tok * a.N + row] = make_float2(yr * f, yi * f);
      }
    }
  }
#endif
}

template <int T, bool EXPORT>
hipError_t launch_pipe(const WlArgs& a, int8_t* xp, hipStream_t s) {
  const int64_t nks = a.K / 64, nfrag = (a.B + 15) / 16;
  const int64_t nchunks = nfrag * nks * 2 * 64;
  int64_t pblocks = (nchunks + 255) / 256;
  if (pblocks > 65536) pblocks = 65536;
  const bool vec = (reinterpret_cast<uintptr_t>(a.x) & 15) == 0;
  hipLaunchKernelGGL(prefill_prep_kernel, dim3((unsigned)pblocks), dim3(256), 0, s,
                     static_cast<const int8_t*>(a.x), a.B, a.K, nks, reinterpret_cast<uint4*>(xp), nchunks, vec);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((unsigned)((a.N + 31) / 32), (unsigned)((nfrag + 3) / 4));
  hipLaunchKernelGGL((gemm_i8_pipe_kernel<T, EXPORT>), grid, dim3(256), 0, s, a, xp);
  return hipGetLastError();
}

template <int T, bool EXPORT>
hipError_t launch_t(const WlArgs& a, hipStream_t s) {
  constexpr int TOKW = (T <= 2) ? 32 : 16;
  const bool aligned = (a.K % 16) == 0;
  dim3 grid((unsigned)((a.N + 31) / 32), (unsigned)((a.B + 2 * TOKW - 1) / (2 * TOKW)));
  hipLaunchKernelGGL((gemm_i8_kernel<T, TOKW, EXPORT>), grid, dim3(256), 0, s, a, aligned);
  return hipGetLastError();
}

template <bool EXPORT>
hipError_t launch_e(const WlArgs& a, void* ws, hipStream_t s) {
  int8_t* xp = static_cast<int8_t*>(ws);
  if (xp && gemm_workspace_bytes(a.N, a.K, a.B) > 0) {
    switch (a.T) {
      case 1: return launch_pipe<1, EXPORT>(a, xp, s);
      case 2: return launch_pipe<2, EXPORT>(a, xp, s);
      case 3: return launch_pipe<3, EXPORT>(a, xp, s);
      default: return launch_pipe<4, EXPORT>(a, xp, s);
    }
  }
  switch (a.T) {
    case 1: return launch_t<1, EXPORT>(a, s);
    case 2: return launch_t<2, EXPORT>(a, s);
    case 3: return launch_t<3, EXPORT>(a, s);
    default: return launch_t<4, EXPORT>(a, s);
  }
}

}  // namespace

size_t gemm_workspace_bytes(int64_t N, int64_t K, int64_t B) {
  // the pipelined kernel: K % 64 == 0 and every buffer offset within 32 bits
  if (K % 64 != 0 || N * K / 4 >= ((int64_t)1 << 31)) return 0;
  const int64_t bytes = (B + 15) / 16 * (K / 64) * 2048;
  if (bytes >= ((int64_t)1 << 31)) return 0;
  return (size_t)bytes;
}

hipError_t launch_gemm_i8(const WlArgs& a, void* workspace, hipStream_t s) {
  return a.acc ? launch_e<true>(a, workspace, s) : launch_e<false>(a, workspace, s);
}

}  // namespace fairy2i
