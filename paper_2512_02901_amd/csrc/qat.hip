// Quantisation-aware training pieces of one widely-linear layer (Sec. 3.2,
// QAT paragraph and remark (iii); Sec. 3.3, the QAT remarks after the formal
// definition):
//   fq_dequant_kernel   fake-quant forward: after the T quantiser stages
//                       (quantize.hip), W^ = sum_t s_t b_t per entry, summed
//                       in double and rounded once to float32 or bf16
//   ste_*_kernel        straight-through backward through the stage
//                       recursion (b(.) with an identity Jacobian, scales
//                       differentiated through their masked means), stages
//                       in reverse order, reductions in a fixed order
//   cgemm_gauss_kernel  complex GEMM with Gauss's three real products,
//                       P1 = Ar Br, P2 = Ai Bi, P3 = (Ar + Ai)(Br + Bi),
//                       C = (P1 - P2) + i (P3 - P1 - P2), on the bf16 matrix
//                       cores with float32 accumulation
#include "common.h"

namespace fairy2i {

namespace {

constexpr int kQatThreads = 256;
constexpr int kQatMaxBlocks = 1024;

// ------------------------------------------------------------ roundings ---
__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// double -> bf16, nearest with ties to even, one rounding (normal range;
// values below the smallest normal bf16 go through float32).
__device__ inline uint16_t f64_to_bf16(double d) {
  const uint64_t u = (uint64_t)__double_as_longlong(d);
  const uint64_t a = u & 0x7FFFFFFFFFFFFFFFull;
  const uint16_t sgn = (uint16_t)((u >> 48) & 0x8000u);
  if (a == 0) return sgn;
  const int e = (int)(a >> 52) - 1023;
  if (e < -126) return f32_to_bf16((float)d);
  // keep 7 of the 52 fraction bits; a carry moves into the exponent
  const uint64_t r = (a + ((1ull << 44) - 1) + ((a >> 45) & 1ull)) >> 45;  // exponent (11 bits) : fraction (7)
  const uint64_t b = r - ((uint64_t)(1023 - 127) << 7);
  return (uint16_t)(b >= 0x7F80u ? 0x7F80u : b) | sgn;
}

// ------------------------------------------------------------ fake quant ---
// One thread per packed byte (four entries of a row): the entries' codes of
// every stage, dequantised with that stage's scales (Eq. ifairy-dequant) and
// summed over the stages in increasing order (Eq. res-sum).
__global__ __launch_bounds__(kQatThreads) void fq_dequant_kernel(const uint8_t* __restrict__ codes,
                                                                 const float* __restrict__ scales, int T,
                                                                 int64_t nbytes, void* __restrict__ out,
                                                                 int out_dtype) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t bi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; bi < nbytes; bi += stride) {
    uint32_t c[FAIRY2I_MAX_STAGES];
    for (int t = 0; t < T; ++t) c[t] = codes[(int64_t)t * nbytes + bi];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      double re = 0.0, im = 0.0;
      for (int t = 0; t < T; ++t) {
        const uint32_t k = (c[t] >> (2 * e)) & 3u;
        const double s_re = (double)scales[2 * t], s_im = (double)scales[2 * t + 1];
        if (k == 0u) re += s_re;
        else if (k == 2u) re -= s_re;
        else if (k == 1u) im += s_im;
        else im -= s_im;
      }
      const int64_t j = 4 * bi + e;
      if (out_dtype == FAIRY2I_ACT_F32) {
        static_cast<float2*>(out)[j] = make_float2((float)re, (float)im);
      } else {
        const uint32_t w = (uint32_t)f64_to_bf16(re) | ((uint32_t)f64_to_bf16(im) << 16);
        static_cast<uint32_t*>(out)[j] = w;
      }
    }
  }
}

// ----------------------------------------------------- STE backward ---
// Stage t of the reverse recursion, with H = dL/dR_{t+1} held in g_master
// (zero before the last stage) and G = dL/dW^:
//   G_Q = G - H;  d_re = sum_j Re G_Q_j b_re_j / n_re,  d_im likewise;
//   H  += (s_re Re G_Q + b_re d_re) + i (s_im Im G_Q + b_im d_im).

struct StePart {
  double sum[2];
  unsigned long long n[2];
};

__device__ inline double block_sum_double(double v, double* sh) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  double s = 0.0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += sh[i];  // fixed order
  return s;
}

__device__ inline unsigned long long block_sum_u64(unsigned long long v, unsigned long long* sh) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  unsigned long long s = 0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += sh[i];
  return s;
}

// Each thread takes units of 16 entries: 4 code bytes (entry e is code
// (byte[e / 4] >> 2 (e % 4)) & 3) and 128 bytes of G and of H, as 16-byte
// loads when G and H are 16-byte aligned (VEC) and the unit is whole; a last,
// partial unit goes one entry at a time.  FIRST: the first stage of the
// reverse recursion, where H is still zero (not read, only written).
template <bool VEC>
__device__ inline int ste_unit(const uint8_t* __restrict__ codes_t, const float2* __restrict__ p, int64_t u,
                               int64_t nelem, uint32_t& c, float2 (&v)[16]) {
  const int64_t e0 = 16 * u;
  const int n = nelem - e0 < 16 ? (int)(nelem - e0) : 16;
  c = 0u;
  for (int b = 0; b < (n + 3) / 4; ++b) c |= (uint32_t)codes_t[4 * u + b] << (8 * b);
  if (VEC && n == 16) {
    const float4* q = reinterpret_cast<const float4*>(p + e0);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float4 f = q[i];
      v[2 * i] = make_float2(f.x, f.y);
      v[2 * i + 1] = make_float2(f.z, f.w);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = i < n ? p[e0 + i] : make_float2(0.0f, 0.0f);
  }
  return n;
}

template <bool VEC>
__device__ inline void ste_h16(const float2* __restrict__ p, int64_t u, int n, float2 (&v)[16]) {
  const int64_t e0 = 16 * u;
  if (VEC && n == 16) {
    const float4* q = reinterpret_cast<const float4*>(p + e0);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float4 f = q[i];
      v[2 * i] = make_float2(f.x, f.y);
      v[2 * i + 1] = make_float2(f.z, f.w);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = i < n ? p[e0 + i] : make_float2(0.0f, 0.0f);
  }
}

template <bool VEC, bool FIRST>
__global__ __launch_bounds__(kQatThreads) void ste_reduce_kernel(const uint8_t* __restrict__ codes_t,
                                                                 const float2* __restrict__ G,
                                                                 const float2* __restrict__ H, int64_t nelem,
                                                                 StePart* __restrict__ part) {
  __shared__ double shd[kQatThreads / 64];
  __shared__ unsigned long long shn[kQatThreads / 64];
  double s_re = 0.0, s_im = 0.0;
  unsigned long long n_re = 0, n_im = 0;
  const int64_t nunits = (nelem + 15) / 16;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < nunits; u += stride) {
    uint32_t c;
    float2 g[16], h[16];
    const int n = ste_unit<VEC>(codes_t, G, u, nelem, c, g);
    if constexpr (!FIRST) ste_h16<VEC>(H, u, n, h);
    // every entry predicated, no early exit: a fully unrolled loop with
    // constant indices keeps g and h in registers
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const uint32_t k = (c >> (2 * e)) & 3u;
      const double gq_re = FIRST ? (double)g[e].x : (double)g[e].x - (double)h[e].x;
      const double gq_im = FIRST ? (double)g[e].y : (double)g[e].y - (double)h[e].y;
      const double sg = (k & 2u) ? -1.0 : 1.0;  // codes 2, 3 are -1, -i
      // selects, not a branch on which sum to bump (that also puts the pair
      // in scratch memory)
      const bool on = e < n, odd = (k & 1u) != 0u;
      s_im = (on && odd) ? s_im + sg * gq_im : s_im;
      s_re = (on && !odd) ? s_re + sg * gq_re : s_re;
      n_im += (on && odd) ? 1ull : 0ull;
      n_re += (on && !odd) ? 1ull : 0ull;
    }
  }
  const double a = block_sum_double(s_re, shd);
  const double b = block_sum_double(s_im, shd);
  const unsigned long long na = block_sum_u64(n_re, shn);
  const unsigned long long nb = block_sum_u64(n_im, shn);
  if (threadIdx.x == 0) {
    part[blockIdx.x].sum[0] = a;
    part[blockIdx.x].sum[1] = b;
    part[blockIdx.x].n[0] = na;
    part[blockIdx.x].n[1] = nb;
  }
}

// NEXT: the update also forms the next (lower) stage's reduction from the H
// it has just written (codes_n: that stage's codes), with the same threads,
// units and order as ste_reduce_kernel, into part_n: one pass over G and H
// instead of two per stage.
template <bool VEC, bool FIRST, bool NEXT>
__global__ __launch_bounds__(kQatThreads) void ste_update_kernel(const uint8_t* __restrict__ codes_t,
                                                                 const float* __restrict__ scales_t,
                                                                 const float2* __restrict__ G,
                                                                 float2* __restrict__ H, int64_t nelem,
                                                                 const StePart* __restrict__ part, int nblk,
                                                                 const uint8_t* __restrict__ codes_n,
                                                                 StePart* __restrict__ part_n) {
  // d[axis] = (sum of the reduction blocks' partial sums) / n, formed by every
  // block alike: thread i sums partials i, i + 256, ... in order, then the
  // block's fixed-order tree, so every block (and every run) gets the same d
  __shared__ double shd[kQatThreads / 64];
  __shared__ unsigned long long shn[kQatThreads / 64];
  double a = 0.0, b = 0.0;
  unsigned long long na = 0, nb = 0;
  for (int i = threadIdx.x; i < nblk; i += blockDim.x) {
    a += part[i].sum[0];
    b += part[i].sum[1];
    na += part[i].n[0];
    nb += part[i].n[1];
  }
  a = block_sum_double(a, shd);
  b = block_sum_double(b, shd);
  na = block_sum_u64(na, shn);
  nb = block_sum_u64(nb, shn);
  const double s_re = (double)scales_t[0], s_im = (double)scales_t[1];
  const double d_re = na ? a / (double)na : 0.0, d_im = nb ? b / (double)nb : 0.0;
  double x_re = 0.0, x_im = 0.0;  // the next stage's sums
  unsigned long long xn_re = 0, xn_im = 0;
  const int64_t nunits = (nelem + 15) / 16;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < nunits; u += stride) {
    uint32_t c, cn = 0u;
    float2 g[16], h[16];
    const int n = ste_unit<VEC>(codes_t, G, u, nelem, c, g);
    if constexpr (NEXT)
      for (int bb = 0; bb < (n + 3) / 4; ++bb) cn |= (uint32_t)codes_n[4 * u + bb] << (8 * bb);
    if constexpr (FIRST) {
#pragma unroll
      for (int e = 0; e < 16; ++e) h[e] = make_float2(0.0f, 0.0f);
    } else {
      ste_h16<VEC>(H, u, n, h);
    }
    float2 o[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const uint32_t k = (c >> (2 * e)) & 3u;
      const double gq_re = (double)g[e].x - (double)h[e].x, gq_im = (double)g[e].y - (double)h[e].y;
      const double sg = (k & 2u) ? -1.0 : 1.0;
      const double b_re = (k & 1u) ? 0.0 : sg;
      const double b_im = (k & 1u) ? sg : 0.0;
      const double nr = (double)h[e].x + (s_re * gq_re + b_re * d_re);
      const double ni = (double)h[e].y + (s_im * gq_im + b_im * d_im);
      o[e] = make_float2((float)nr, (float)ni);
      if constexpr (NEXT) {
        // the next stage's G_Q from the stored (float32) H, as its own reduction would read it
        if (e < n) {
          const uint32_t kn = (cn >> (2 * e)) & 3u;
          const double sn = (kn & 2u) ? -1.0 : 1.0;
          if (kn & 1u) {
            x_im += sn * ((double)g[e].y - (double)o[e].y);
            ++xn_im;
          } else {
            x_re += sn * ((double)g[e].x - (double)o[e].x);
            ++xn_re;
          }
        }
      }
    }
    if (VEC && n == 16) {
      float4* q = reinterpret_cast<float4*>(H + 16 * u);
#pragma unroll
      for (int i = 0; i < 8; ++i) q[i] = make_float4(o[2 * i].x, o[2 * i].y, o[2 * i + 1].x, o[2 * i + 1].y);
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (e < n) H[16 * u + e] = o[e];  // constant indices: o stays in registers
    }
  }
  if constexpr (NEXT) {
    const double xa = block_sum_double(x_re, shd);
    const double xb = block_sum_double(x_im, shd);
    const unsigned long long xna = block_sum_u64(xn_re, shn);
    const unsigned long long xnb = block_sum_u64(xn_im, shn);
    if (threadIdx.x == 0) {
      part_n[blockIdx.x].sum[0] = xa;
      part_n[blockIdx.x].sum[1] = xb;
      part_n[blockIdx.x].n[0] = xna;
      part_n[blockIdx.x].n[1] = xnb;
    }
  }
}

int qat_blocks(int64_t nbytes) {
  int64_t b = (nbytes + kQatThreads - 1) / kQatThreads;
  if (b > kQatMaxBlocks) b = kQatMaxBlocks;
  if (b < 1) b = 1;
  return (int)b;
}

// ------------------------------------------------------- Gauss GEMM ---
// C[m][n] (+)= sum over segments s and k < K_s of opA_s(m, k) * opB_s(n, k):
// an operand holds `rows` x K complex values, either row-major with K
// contiguous (trans = 0, element (r, k) at r ld + k) or with the rows
// contiguous (trans = 1, element (r, k) at k ld + r), as float32 or bf16
// pairs; conj negates its imaginary parts.  Block tile 64 x 64 of C, four
// waves of 32 x 32, 32 values of k per step.  Each step stages three bf16
// planes per operand in LDS: Re, Im and Re + Im (the sum formed in float32
// from the inputs and rounded once), and each wave runs the three real
// products on v_mfma_f32_16x16x32_bf16 into float32 accumulators:
//     P1 = Ar Br,   P2 = Ai Bi,   P3 = (Ar + Ai)(Br + Bi),
//     C = (P1 - P2) + i (P3 - P1 - P2).
constexpr int kGT = 64;    // block tile rows / columns
constexpr int kGK = 32;    // k per step
constexpr int kGRow = 40;  // LDS row stride in bf16 (80 bytes: 16-byte aligned rows)

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct GemmOp {
  const void* p;
  int64_t ld;
  int32_t dtype, trans, conj, pad_;
};

struct GemmArgs {
  GemmOp a[2], b[2];
  int64_t K[2];
  int64_t M, N, ldc;
  float2* C;
  int32_t nseg, accumulate;
};

// Eight consecutive complex values of an operand along its contiguous
// dimension, starting at element index `base`; only the first `nv` exist
// (the rest read as zero).
__device__ inline void load8(const GemmOp& op, int64_t base, int nv, float (&re)[8], float (&im)[8]) {
  if (op.dtype == FAIRY2I_ACT_BF16) {
    const uint32_t* src = static_cast<const uint32_t*>(op.p) + base;
    uint32_t w[8];
    if (nv == 8 && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
      const uint4 v0 = reinterpret_cast<const uint4*>(src)[0], v1 = reinterpret_cast<const uint4*>(src)[1];
      w[0] = v0.x; w[1] = v0.y; w[2] = v0.z; w[3] = v0.w;
      w[4] = v1.x; w[5] = v1.y; w[6] = v1.z; w[7] = v1.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) w[e] = e < nv ? src[e] : 0u;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      re[e] = __uint_as_float(w[e] << 16);
      im[e] = __uint_as_float(w[e] & 0xFFFF0000u);
    }
  } else {
    const float2* src = static_cast<const float2*>(op.p) + base;
    if (nv == 8 && (reinterpret_cast<uintptr_t>(src) & 15) == 0) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 v = reinterpret_cast<const float4*>(src)[q];
        re[2 * q] = v.x; im[2 * q] = v.y; re[2 * q + 1] = v.z; im[2 * q + 1] = v.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float2 v = e < nv ? src[e] : make_float2(0.0f, 0.0f);
        re[e] = v.x;
        im[e] = v.y;
      }
    }
  }
  if (op.conj) {
#pragma unroll
    for (int e = 0; e < 8; ++e) im[e] = -im[e];
  }
}

// One operand's 64 x 32 tile (rows r0.., k k0..) into its three LDS planes.
__device__ inline void stage_tile(const GemmOp& op, int64_t rows, int64_t Kseg, int64_t r0, int64_t k0,
                                  uint16_t (*plane)[kGT][kGRow]) {
  const int t = threadIdx.x;
  float re[8], im[8];
  if (!op.trans) {
    const int r = t >> 2, kk = (t & 3) * 8;
    const int64_t gr = r0 + r, gk = k0 + kk;
    int nv = 0;
    if (gr < rows && gk < Kseg) nv = Kseg - gk < 8 ? (int)(Kseg - gk) : 8;
    load8(op, nv ? gr * op.ld + gk : 0, nv, re, im);
    uint32_t pr[4], pi[4], ps[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      pr[q] = (uint32_t)f32_to_bf16(re[2 * q]) | ((uint32_t)f32_to_bf16(re[2 * q + 1]) << 16);
      pi[q] = (uint32_t)f32_to_bf16(im[2 * q]) | ((uint32_t)f32_to_bf16(im[2 * q + 1]) << 16);
      ps[q] = (uint32_t)f32_to_bf16(re[2 * q] + im[2 * q]) | ((uint32_t)f32_to_bf16(re[2 * q + 1] + im[2 * q + 1]) << 16);
    }
    *reinterpret_cast<uint4*>(&plane[0][r][kk]) = make_uint4(pr[0], pr[1], pr[2], pr[3]);
    *reinterpret_cast<uint4*>(&plane[1][r][kk]) = make_uint4(pi[0], pi[1], pi[2], pi[3]);
    *reinterpret_cast<uint4*>(&plane[2][r][kk]) = make_uint4(ps[0], ps[1], ps[2], ps[3]);
  } else {
    const int kk = t >> 3, r = (t & 7) * 8;
    const int64_t gr = r0 + r, gk = k0 + kk;
    int nv = 0;
    if (gk < Kseg && gr < rows) nv = rows - gr < 8 ? (int)(rows - gr) : 8;
    load8(op, nv ? gk * op.ld + gr : 0, nv, re, im);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      plane[0][r + e][kk] = f32_to_bf16(re[e]);
      plane[1][r + e][kk] = f32_to_bf16(im[e]);
      plane[2][r + e][kk] = f32_to_bf16(re[e] + im[e]);
    }
  }
}

__global__ __launch_bounds__(256) void cgemm_gauss_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) uint16_t As[3][kGT][kGRow];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[3][kGT][kGRow];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t m0 = (int64_t)blockIdx.y * kGT, n0 = (int64_t)blockIdx.x * kGT;
  f32x4 acc[3][2][2];
#pragma unroll
  for (int p = 0; p < 3; ++p)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[p][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15, fk = (lane >> 4) * 8;  // fragment row and first k of this lane
  for (int s = 0; s < g.nseg; ++s) {
    const GemmOp A = g.a[s], B = g.b[s];
    const int64_t Ks = g.K[s];
    for (int64_t k0 = 0; k0 < Ks; k0 += kGK) {
      __syncthreads();
      stage_tile(A, g.M, Ks, m0, k0, As);
      stage_tile(B, g.N, Ks, n0, k0, Bs);
      __syncthreads();
      bf16x8 fa[3][2], fb[3][2];
#pragma unroll
      for (int p = 0; p < 3; ++p)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          fa[p][i] = *reinterpret_cast<const bf16x8*>(&As[p][32 * wm + 16 * i + fr][fk]);
          fb[p][i] = *reinterpret_cast<const bf16x8*>(&Bs[p][32 * wn + 16 * i + fr][fk]);
        }
#pragma unroll
      for (int p = 0; p < 3; ++p)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[p][i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[p][i], fb[p][j], acc[p][i][j], 0, 0, 0);
    }
  }
  // lane holds C rows 4 (lane / 16) + q of column lane % 16 of each 16 x 16 tile
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t n = n0 + 32 * wn + 16 * j + fr;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int64_t m = m0 + 32 * wm + 16 * i + 4 * (lane >> 4) + q;
        if (m < g.M && n < g.N) {
          const float p1 = acc[0][i][j][q], p2 = acc[1][i][j][q], p3 = acc[2][i][j][q];
          float2 v = make_float2(p1 - p2, (p3 - p1) - p2);
          float2* dst = g.C + m * g.ldc + n;
          if (g.accumulate) {
            const float2 o = *dst;
            v = make_float2(o.x + v.x, o.y + v.y);
          }
          *dst = v;
        }
      }
    }
}

bool op_ok(const fairy2i_cgemm_operand& o, int64_t rows, int64_t K) {
  if (!o.data) return false;
  if (o.dtype != FAIRY2I_ACT_F32 && o.dtype != FAIRY2I_ACT_BF16) return false;
  if ((o.trans != 0 && o.trans != 1) || (o.conj != 0 && o.conj != 1) || o.reserved != 0) return false;
  return o.trans ? o.ld >= rows : o.ld >= K;
}

}  // namespace

}  // namespace fairy2i

using namespace fairy2i;

namespace {
inline hipStream_t qat_stream(void* s) { return static_cast<hipStream_t>(s); }
inline fairy2i_status qat_status(hipError_t e) { return e == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP; }
}  // namespace

extern "C" {

fairy2i_status fairy2i_qat_fake_quant(const float* M, int64_t N, int64_t K, int32_t T, uint8_t* codes,
                                      float* scales, void* w_hat, int32_t out_dtype, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  if (!M || !codes || !scales || !w_hat) return FAIRY2I_ERR_NULL;
  if (N <= 0 || K <= 0 || (K % 4) != 0 || N > FAIRY2I_MAX_QUANTIZE_ENTRIES / K) return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (out_dtype != FAIRY2I_ACT_F32 && out_dtype != FAIRY2I_ACT_BF16) return FAIRY2I_ERR_DTYPE;
  if (!workspace || workspace_bytes < quantize_workspace_bytes(N, K)) return FAIRY2I_ERR_WORKSPACE;
  const hipStream_t s = qat_stream(stream);
  hipError_t e = launch_quantize(reinterpret_cast<const float2*>(M), N, K, T, codes, scales, workspace, s);
  if (e != hipSuccess) return FAIRY2I_ERR_HIP;
  const int64_t nbytes = N * K / 4;
  hipLaunchKernelGGL(fq_dequant_kernel, dim3(qat_blocks(nbytes)), dim3(kQatThreads), 0, s, codes, scales, T, nbytes,
                     w_hat, out_dtype);
  return qat_status(hipGetLastError());
}

size_t fairy2i_qat_ste_workspace_bytes(int64_t N, int64_t K) {
  if (N <= 0 || K <= 0 || (K % 4) != 0) return 0;
  return 2 * (size_t)qat_blocks((N * K + 15) / 16) * sizeof(StePart);  // this stage's partials and the next's
}

fairy2i_status fairy2i_qat_ste_backward(const uint8_t* codes, const float* scales, int32_t T, int64_t N, int64_t K,
                                        const float* g_hat, float* g_master, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  if (!codes || !scales || !g_hat || !g_master) return FAIRY2I_ERR_NULL;
  if (N <= 0 || K <= 0 || (K % 4) != 0 || N > FAIRY2I_MAX_QUANTIZE_ENTRIES / K) return FAIRY2I_ERR_SHAPE;
  if (T < 1 || T > FAIRY2I_MAX_STAGES) return FAIRY2I_ERR_STAGES;
  if (!workspace || workspace_bytes < fairy2i_qat_ste_workspace_bytes(N, K)) return FAIRY2I_ERR_WORKSPACE;
  const hipStream_t s = qat_stream(stream);
  const int64_t nelem = N * K, nbytes = nelem / 4;
  const int nblk = qat_blocks((nelem + 15) / 16);
  auto* part = static_cast<StePart*>(workspace);
  const auto* G = reinterpret_cast<const float2*>(g_hat);
  auto* H = reinterpret_cast<float2*>(g_master);
  const bool vec = ((reinterpret_cast<uintptr_t>(g_hat) | reinterpret_cast<uintptr_t>(g_master)) & 15) == 0;
  hipError_t e = hipSuccess;
  // the last stage's reduction reads G only (H is still zero); every update
  // but the first stage's also forms the next stage's reduction
  StePart* cur = part;
  StePart* nxt = part + nblk;
  {
    const uint8_t* ct = codes + (int64_t)(T - 1) * nbytes;
    if (vec) hipLaunchKernelGGL((ste_reduce_kernel<true, true>), dim3(nblk), dim3(kQatThreads), 0, s, ct, G, H, nelem, cur);
    else hipLaunchKernelGGL((ste_reduce_kernel<false, true>), dim3(nblk), dim3(kQatThreads), 0, s, ct, G, H, nelem, cur);
    e = hipGetLastError();
  }
  for (int t = T - 1; t >= 0 && e == hipSuccess; --t) {
    const uint8_t* ct = codes + (int64_t)t * nbytes;
    const uint8_t* cn = t > 0 ? codes + (int64_t)(t - 1) * nbytes : nullptr;
    const bool first = t == T - 1;  // H is still zero: not read, only written
    const bool next = t > 0;
    using K = void (*)(const uint8_t*, const float*, const float2*, float2*, int64_t, const StePart*, int,
                       const uint8_t*, StePart*);
    const K kernels[2][2][2] = {
        {{ste_update_kernel<false, false, false>, ste_update_kernel<false, false, true>},
         {ste_update_kernel<false, true, false>, ste_update_kernel<false, true, true>}},
        {{ste_update_kernel<true, false, false>, ste_update_kernel<true, false, true>},
         {ste_update_kernel<true, true, false>, ste_update_kernel<true, true, true>}}};
    hipLaunchKernelGGL(kernels[vec][first][next], dim3(nblk), dim3(kQatThreads), 0, s, ct, scales + 2 * t, G, H,
                       nelem, cur, nblk, cn, nxt);
    e = hipGetLastError();
    StePart* tmp = cur;
    cur = nxt;
    nxt = tmp;
  }
  return qat_status(e);
}

fairy2i_status fairy2i_cgemm_gauss(const fairy2i_cgemm_operand* A, const fairy2i_cgemm_operand* B, const int64_t* K,
                                   int32_t nseg, int64_t M, int64_t N, float* C, int64_t ldc, int32_t accumulate,
                                   void* stream) {
  if (!A || !B || !K || !C) return FAIRY2I_ERR_NULL;
  if (nseg < 1 || nseg > 2 || M <= 0 || N <= 0 || ldc < N || (accumulate != 0 && accumulate != 1))
    return FAIRY2I_ERR_SHAPE;
  if (M > 65535LL * kGT || N > ((int64_t)1 << 31)) return FAIRY2I_ERR_UNSUPPORTED;
  GemmArgs g{};
  for (int s = 0; s < nseg; ++s) {
    if (K[s] <= 0) return FAIRY2I_ERR_SHAPE;
    if (!A[s].data || !B[s].data) return FAIRY2I_ERR_NULL;
    if (!op_ok(A[s], M, K[s]) || !op_ok(B[s], N, K[s])) return FAIRY2I_ERR_SHAPE;
    g.a[s] = GemmOp{A[s].data, A[s].ld, A[s].dtype, A[s].trans, A[s].conj, 0};
    g.b[s] = GemmOp{B[s].data, B[s].ld, B[s].dtype, B[s].trans, B[s].conj, 0};
    g.K[s] = K[s];
  }
  g.nseg = nseg;
  g.M = M;
  g.N = N;
  g.ldc = ldc;
  g.C = reinterpret_cast<float2*>(C);
  g.accumulate = accumulate;
  const dim3 grid((unsigned)((N + kGT - 1) / kGT), (unsigned)((M + kGT - 1) / kGT));
  hipLaunchKernelGGL(cgemm_gauss_kernel, grid, dim3(256), 0, qat_stream(stream), g);
  return qat_status(hipGetLastError());
}

}  // extern "C"
