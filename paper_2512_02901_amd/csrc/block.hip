// One widely-linear decoder block for one decode token (Sec. 1: every linear
// layer of the LLaMA-style block becomes a widely-linear layer; Sec. 3.1,
// self-attention paragraph, Eq. hermitian-score: scores Re(q^H k) / sqrt(d_k),
// softmax and value aggregation acting on the real and imaginary parts alike,
// a widely-linear output projection).
//
// The seven projections run on the grouped fp8 x fp4 decode path (q, k, v in
// one call; o; gate and up in one call; down).  Between them:
//   add_rmsnorm   residual add, RMSNorm over the 2n real components, bf16 out
//   rope_append   rotary embedding as a complex rotation per head entry
//                 (angles in double), key and value written to the caches
//   attn_partial  per (head, 64-position slice): scores, slice max, slice
//                 softmax sum and the slice's weighted sum of values
//   attn_combine  the slices of a head merged in slice order, bf16 out
//   swiglu        silu(Re g) Re u + i silu(Im g) Im u, bf16 out
//   add           the final residual add
// For one token on the fp4 path with two digit bands (every block this
// library plans, up to 8192 complex entries per token) the fused path runs
// instead: 13 launches in place of 19.  The stage that consumes a
// projection's output sums that projection's split-K partials itself, and
// the stage that makes a projection's input writes its activation operand:
//   operand (norm)  x (+ the o projection's output), RMSNorm, operand of
//                   q k v (of gate and up)
//   rope_append_sum q k v summed, rotary embedding, caches
//   operand (bf16)  operand of a bf16 token (the attention output; SwiGLU's)
//   swiglu_sum      gate and up summed, SwiGLU, bf16 out
//   add_sum         down summed, the final residual add
// so only the product kernels of the four group calls remain of them.
// Complex vectors are float2 (re, im); a head owns dc = n / n_heads
// consecutive complex entries (entry j: its real dims j and j + dc).  All
// reductions run in a fixed order, so results are bitwise reproducible.
#include <math.h>
#include <string.h>

#include "common.h"
#include "decode.h"
#include "f4_operand.h"

namespace fairy2i {

namespace {

constexpr int kAttnSlice = 64;   // positions per attention slice (one per lane)
constexpr int kMaxAttnSlices = 4096;  // slices per head the combine keeps in LDS
constexpr int kNormThreads = 256;

__device__ inline uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline float wave_sum(float v) {
  // butterfly: every lane ends with the same, commutatively formed sum
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ inline float wave_max(float v) {
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// v = x (+ a); h_out = v (if given); z = bf16(v / sqrt(mean(v^2) + eps) * gamma)
// over the 2n real components.  One block per token.
__global__ __launch_bounds__(kNormThreads) void add_rmsnorm_kernel(const float2* __restrict__ x,
                                                                   const float2* __restrict__ a,
                                                                   float2* __restrict__ h_out,
                                                                   const float* __restrict__ gamma, float eps,
                                                                   int n, uint16_t* __restrict__ z) {
  __shared__ float red[kNormThreads / 64];
  float ss = 0.0f;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    float2 v = x[i];
    if (a) {
      const float2 w = a[i];
      v.x += w.x;
      v.y += w.y;
    }
    ss = fmaf(v.x, v.x, ss);
    ss = fmaf(v.y, v.y, ss);
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float tot = 0.0f;
  for (int w = 0; w < kNormThreads / 64; ++w) tot += red[w];
  const float r = 1.0f / sqrtf(tot / (float)(2 * n) + eps);
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    float2 v = x[i];
    if (a) {
      const float2 w = a[i];
      v.x += w.x;
      v.y += w.y;
    }
    if (h_out) h_out[i] = v;
    z[2 * i] = bf16_rne((v.x * r) * gamma[i]);
    z[2 * i + 1] = bf16_rne((v.y * r) * gamma[n + i]);
  }
}

// Rotary embedding of q and k (entry j of a head turned by pos * theta_j,
// theta_j = base^(-2 j / dh), dh = 2 dc), then k and v stored at position pos
// of the caches [H][max_ctx][dc].
__global__ void rope_append_kernel(const float2* __restrict__ q, const float2* __restrict__ k,
                                   const float2* __restrict__ v, int n, int dc, int64_t pos, int64_t max_ctx,
                                   double base, float2* __restrict__ q_rot, float2* __restrict__ k_cache,
                                   float2* __restrict__ v_cache) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int h = i / dc, j = i - h * dc;
  const double ang = (double)pos * pow(base, -2.0 * (double)j / (double)(2 * dc));
  double s, c;
  sincos(ang, &s, &c);
  const float cf = (float)c, sf = (float)s;
  const float2 qv = q[i], kv = k[i];
  q_rot[i] = make_float2(fmaf(qv.x, cf, -qv.y * sf), fmaf(qv.x, sf, qv.y * cf));
  const int64_t at = ((int64_t)h * max_ctx + pos) * dc + j;
  k_cache[at] = make_float2(fmaf(kv.x, cf, -kv.y * sf), fmaf(kv.x, sf, kv.y * cf));
  v_cache[at] = v[i];
}

// One block of four waves per (64-position slice, head).  Scores: four lanes
// per position, each taking a quarter of the key row's 16-byte chunks (eight
// loads in flight), summed across the four lanes, times scale; then the
// slice's maximum m, e_t = exp(s_t - m) (kept in LDS) and l = sum e_t.
// Values: wave w takes positions 16 w .. 16 w + 15, lane j (+ 64 r) entry j
// of o = sum_t e_t v_t (eight value loads in flight), and the four waves'
// sums are added in wave order.  Partial record per (head, slice):
// [m, l, o (2 dc floats)].
constexpr int kAttnThreads = 256;
template <int R>  // complex entries per lane in the value pass: dc <= 64 R
__global__ __launch_bounds__(kAttnThreads) void attn_partial_kernel(const float2* __restrict__ q_rot,
                                                                    const float2* __restrict__ k_cache,
                                                                    const float2* __restrict__ v_cache, int dc,
                                                                    int64_t n_ctx, int64_t max_ctx, float scale,
                                                                    float* __restrict__ part) {
  __shared__ float es[kAttnSlice];
  __shared__ float redm[kAttnThreads / 64], redl[kAttnThreads / 64];
  __shared__ float2 ow[kAttnThreads / 64][64 * R];
  const int h = blockIdx.y, sl = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t n0 = (int64_t)sl * kAttnSlice;
  const int cnt = (int)min((int64_t)kAttnSlice, n_ctx - n0);
  const float2* kh = k_cache + (int64_t)h * max_ctx * dc;
  const float2* vh = v_cache + (int64_t)h * max_ctx * dc;
  const float4* qh = reinterpret_cast<const float4*>(q_rot + (int64_t)h * dc);
  const int p = tid >> 2, qd = tid & 3, nf4 = dc / 2;
  float acc = 0.0f;
  if (p < cnt) {
    const float4* kp = reinterpret_cast<const float4*>(kh + (n0 + p) * dc);
    for (int j0 = qd; j0 < nf4; j0 += 32) {
      float4 kv[8], qv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int j = j0 + 4 * u;
        kv[u] = j < nf4 ? kp[j] : make_float4(0.f, 0.f, 0.f, 0.f);
        qv[u] = j < nf4 ? qh[j] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        acc = fmaf(qv[u].x, kv[u].x, acc);
        acc = fmaf(qv[u].y, kv[u].y, acc);
        acc = fmaf(qv[u].z, kv[u].z, acc);
        acc = fmaf(qv[u].w, kv[u].w, acc);
      }
    }
  }
  acc += __shfl_xor(acc, 1);
  acc += __shfl_xor(acc, 2);
  const float s = p < cnt ? acc * scale : -INFINITY;
  float m = wave_max(s);
  if (lane == 0) redm[wave] = m;
  __syncthreads();
  m = fmaxf(fmaxf(redm[0], redm[1]), fmaxf(redm[2], redm[3]));
  const float e = p < cnt ? expf(s - m) : 0.0f;
  if (qd == 0) es[p] = e;
  const float lw = wave_sum(qd == 0 ? e : 0.0f);
  if (lane == 0) redl[wave] = lw;
  __syncthreads();
  const float l = ((redl[0] + redl[1]) + redl[2]) + redl[3];
  float2 o[R];
#pragma unroll
  for (int r = 0; r < R; ++r) o[r] = make_float2(0.f, 0.f);
  const int pb = 16 * wave;
#pragma unroll
  for (int t0 = 0; t0 < 16; t0 += 8) {
    float2 vv[8][R];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int t = pb + t0 + u, j = lane + 64 * r;
        vv[u][r] = (t < cnt && j < dc) ? vh[(n0 + t) * dc + j] : make_float2(0.f, 0.f);
      }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float w = es[pb + t0 + u];  // 0 past cnt
#pragma unroll
      for (int r = 0; r < R; ++r) {
        o[r].x = fmaf(w, vv[u][r].x, o[r].x);
        o[r].y = fmaf(w, vv[u][r].y, o[r].y);
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) ow[wave][lane + 64 * r] = o[r];
  __syncthreads();
  float* rec = part + ((int64_t)h * gridDim.x + sl) * (2 + 2 * dc);
  if (tid == 0) {
    rec[0] = m;
    rec[1] = l;
  }
  for (int j = tid; j < dc; j += kAttnThreads) {
    float2 a = ow[0][j];
    for (int w = 1; w < kAttnThreads / 64; ++w) {
      a.x += ow[w][j].x;
      a.y += ow[w][j].y;
    }
    rec[2 + 2 * j] = a.x;
    rec[3 + 2 * j] = a.y;
  }
}

// Per head: M = max_s m_s, f_s = e^(m_s - M) (kept in LDS), L = sum_s l_s f_s,
// o_j = sum_s o_{s,j} f_s / L over the slices in order; written as bf16 pairs
// at the head's entries.
__global__ __launch_bounds__(64) void attn_combine_kernel(const float* __restrict__ part, int n_slices, int dc,
                                                          uint16_t* __restrict__ o_out) {
  __shared__ float fs[kMaxAttnSlices];
  const int h = blockIdx.x, lane = threadIdx.x;
  const int rl = 2 + 2 * dc;
  const float* ph = part + (int64_t)h * n_slices * rl;
  float M = -INFINITY;
  for (int sl = lane; sl < n_slices; sl += 64) M = fmaxf(M, ph[(int64_t)sl * rl]);
  M = wave_max(M);
  float L = 0.0f;
  for (int s0 = 0; s0 < n_slices; s0 += 64) {
    const int sl = s0 + lane;
    float f = 0.0f, t = 0.0f;
    if (sl < n_slices) {
      f = expf(ph[(int64_t)sl * rl] - M);
      t = ph[(int64_t)sl * rl + 1] * f;
      fs[sl] = f;
    }
    L += wave_sum(t);
  }
  __syncthreads();
  const float invL = 1.0f / L;
  for (int j = lane; j < dc; j += 64) {
    float ore = 0.0f, oim = 0.0f;
    for (int s0 = 0; s0 < n_slices; s0 += 8) {
      float2 ov[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        ov[u] = s0 + u < n_slices ? *reinterpret_cast<const float2*>(ph + (int64_t)(s0 + u) * rl + 2 + 2 * j)
                                  : make_float2(0.f, 0.f);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float f = s0 + u < n_slices ? fs[s0 + u] : 0.0f;
        ore = fmaf(ov[u].x, f, ore);
        oim = fmaf(ov[u].y, f, oim);
      }
    }
    o_out[2 * (h * dc + j)] = bf16_rne(ore * invL);
    o_out[2 * (h * dc + j) + 1] = bf16_rne(oim * invL);
  }
}

__device__ inline float silu(float v) { return v / (1.0f + expf(-v)); }

__global__ void swiglu_kernel(const float2* __restrict__ g, const float2* __restrict__ u, int n,
                              uint16_t* __restrict__ act) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float2 gv = g[i], uv = u[i];
  act[2 * i] = bf16_rne(silu(gv.x) * uv.x);
  act[2 * i + 1] = bf16_rne(silu(gv.y) * uv.y);
}

__global__ void add_kernel(const float2* __restrict__ a, const float2* __restrict__ b, int n,
                           float2* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const float2 av = a[i], bv = b[i];
  out[i] = make_float2(av.x + bv.x, av.y + bv.y);
}

// ---------------------------------------------------------- fused path ---
// For one token on the fp4 path (two digit bands, one 8-column tile), the
// block's elementwise stages also do the grouped call's other two launches:
// the kernel that needs a layer's output sums that layer's split-K partials
// itself (in slice order, the additions of the grouped call's reduction),
// and the stage that makes a projection's input also writes that
// projection's activation operand (token shift, digit pairs; f4_operand.h).

// A projection's output: its split-K partials [nkc][N] or, with one slice,
// the output itself.
struct LayerOut {
  const float2* part;
  float2* y;
  int32_t nkc, N;
};

// Entry i of NS projections' outputs: each output's slices added in order
// from +0 (the additions of the grouped call's reduction), the loads of U
// slices of every output in flight together; summed outputs are also written
// where that reduction would write them.
template <int NS, int U = 8>
__device__ inline void layer_outs(const LayerOut (&o)[NS], int i, float2 (&r)[NS]) {
  int mk = 1;
#pragma unroll
  for (int q = 0; q < NS; ++q) {
    mk = max(mk, o[q].nkc);
    r[q] = make_float2(0.0f, 0.0f);
  }
  for (int kc0 = 0; kc0 < mk; kc0 += U) {
    float2 t[NS][U];
#pragma unroll
    for (int q = 0; q < NS; ++q)
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int kc = kc0 + u;
        t[q][u] = o[q].nkc > 1 ? (kc < o[q].nkc ? o[q].part[(int64_t)kc * o[q].N + i] : make_float2(0.f, 0.f))
                               : (kc == 0 ? o[q].y[i] : make_float2(0.f, 0.f));
      }
#pragma unroll
    for (int q = 0; q < NS; ++q)
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (kc0 + u < max(o[q].nkc, 1)) {
          r[q].x += t[q][u].x;
          r[q].y += t[q][u].y;
        }
  }
#pragma unroll
  for (int q = 0; q < NS; ++q)
    if (o[q].nkc > 1) o[q].y[i] = r[q];
}

// Up to three projections fed the same token: their operand buffers and
// output factors, the operand's 256-code steps and the claim counter of
// their group call (zeroed for the product kernel, as the grouped call's
// own operand kernel does).
struct OperandTargets {
  int8_t* xf[3];
  float* xs[3];
  int32_t count, nk4;
  uint32_t* ctr;
};

constexpr int kOpThreads = 512;
constexpr int kOpMaxK = 16 * kOpThreads;  // complex entries of a token the operand kernel takes
constexpr int kSrcNorm = 0, kSrcBf16 = 1;

struct OperandArgs {
  int32_t K;  // complex entries of the token
  // kSrcNorm: v = x (+ the residual branch res); h_out = v; z = RMSNorm(v) gamma
  const float2* x;
  LayerOut res;      // res.y null: no residual branch
  float2* h_out;
  const float* gamma;
  float eps;
  uint16_t* z_out;  // the bf16 token
  // kSrcBf16: the token as bf16 (re, im) words
  const uint32_t* tok;
  OperandTargets t;
};

// Entries tid + e kOpThreads (e < E) of a projection's output, every load of
// U slices in flight together; the slices are added in order.
template <int E>
__device__ inline void gather_out(const LayerOut& o, int tid, int K, float2 (&acc)[E]) {
  constexpr int U = E <= 4 ? 8 : (E <= 8 ? 4 : 2);
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = make_float2(0.0f, 0.0f);
  if (o.nkc <= 1) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = tid + e * kOpThreads;
      if (i < K) acc[e] = o.y[i];
    }
    return;
  }
  for (int kc0 = 0; kc0 < o.nkc; kc0 += U) {
    float2 t[U][E];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int i = tid + e * kOpThreads;
        t[u][e] = (kc0 + u < o.nkc && i < K) ? o.part[(int64_t)(kc0 + u) * o.N + i] : make_float2(0.0f, 0.0f);
      }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (kc0 + u < o.nkc)
#pragma unroll
        for (int e = 0; e < E; ++e) {
          acc[e].x += t[u][e].x;
          acc[e].y += t[u][e].y;
        }
  }
  // the sums start from +0 and add the slices in order, as the grouped
  // call's reduction does; write them where that reduction would
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = tid + e * kOpThreads;
    if (i < K) o.y[i] = acc[e];
  }
}

// One block: the token's bf16 words in LDS (entry i of thread i mod
// kOpThreads, E entries a thread: K <= E kOpThreads), their largest
// magnitude, then the digits of every half run (8 codes) of the operand
// (runs past K hold zeros) for each target.
template <int SRC, int E>
__global__ __launch_bounds__(kOpThreads) void block_operand_kernel(OperandArgs a) {
  __shared__ __align__(16) uint32_t tokw[E * kOpThreads];
  __shared__ float red[kOpThreads / 64];
  __shared__ float sh_g;
  const int K = a.K, tid = threadIdx.x, wave = tid >> 6;
  uint32_t zw[E];
  if constexpr (SRC == kSrcNorm) {
    float2 v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = tid + e * kOpThreads;
      v[e] = i < K ? a.x[i] : make_float2(0.0f, 0.0f);
    }
    if (a.res.y) {
      float2 w[E];
      gather_out<E>(a.res, tid, K, w);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        v[e].x += w[e].x;
        v[e].y += w[e].y;
      }
    }
    float ss = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      ss = fmaf(v[e].x, v[e].x, ss);
      ss = fmaf(v[e].y, v[e].y, ss);
    }
    ss = wave_sum(ss);
    if ((tid & 63) == 0) red[wave] = ss;
    __syncthreads();
    float tot = 0.0f;
    for (int w = 0; w < kOpThreads / 64; ++w) tot += red[w];
    const float r = 1.0f / sqrtf(tot / (float)(2 * K) + a.eps);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = tid + e * kOpThreads;
      zw[e] = 0u;
      if (i < K) {
        if (a.h_out) a.h_out[i] = v[e];
        zw[e] = (uint32_t)bf16_rne((v[e].x * r) * a.gamma[i]) | ((uint32_t)bf16_rne((v[e].y * r) * a.gamma[K + i]) << 16);
      }
    }
    __syncthreads();  // red is reused below
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int i = tid + e * kOpThreads;
      zw[e] = i < K ? a.tok[i] : 0u;
    }
  }
  float m = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = tid + e * kOpThreads;
    if (i < K) {
      tokw[i] = zw[e];
      if constexpr (SRC == kSrcNorm) reinterpret_cast<uint32_t*>(a.z_out)[i] = zw[e];
      m = fmaxf(m, fmaxf(fabsf(__uint_as_float(zw[e] << 16)), fabsf(__uint_as_float(zw[e] & 0xFFFF0000u))));
    }
  }
  m = wave_max(m);
  if ((tid & 63) == 0) red[wave] = m;
  __syncthreads();
  if (tid == 0) {
    float g = 0.0f;
    for (int w = 0; w < kOpThreads / 64; ++w) g = fmaxf(g, red[w]);
    sh_g = g;
  }
  __syncthreads();
  const float g = sh_g;
  const int S = f4_token_shift(g);
  if (tid == 0) {
    for (int t = 0; t < a.t.count; ++t) a.t.xs[t][0] = g > 0.0f ? ldexpf(1.0f, -S) : 0.0f;
    if (a.t.ctr) *a.t.ctr = 0u;
  }
  uint8_t* const dst[3] = {reinterpret_cast<uint8_t*>(a.t.xf[0]), reinterpret_cast<uint8_t*>(a.t.xf[1]),
                           reinterpret_cast<uint8_t*>(a.t.xf[2])};
  f4_encode_token<kOpThreads, 3>(tokw, K, S, a.t.nk4, dst, a.t.count);
}

template <int SRC>
void launch_operand(const OperandArgs& a, hipStream_t s) {
  const dim3 g(1), b(kOpThreads);
  if (a.K <= 4 * kOpThreads) hipLaunchKernelGGL((block_operand_kernel<SRC, 4>), g, b, 0, s, a);
  else if (a.K <= 8 * kOpThreads) hipLaunchKernelGGL((block_operand_kernel<SRC, 8>), g, b, 0, s, a);
  else hipLaunchKernelGGL((block_operand_kernel<SRC, 16>), g, b, 0, s, a);
}

// rope_append_kernel on the summed q, k and v partials (also written out).
__global__ void rope_append_sum_kernel(LayerOut q, LayerOut k, LayerOut v, int n, int dc, int64_t pos,
                                       int64_t max_ctx, double base, float2* __restrict__ q_rot,
                                       float2* __restrict__ k_cache, float2* __restrict__ v_cache) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const LayerOut o[3] = {q, k, v};
  float2 r[3];
  layer_outs<3>(o, i, r);
  const float2 qv = r[0], kv = r[1], vv = r[2];
  const int h = i / dc, j = i - h * dc;
  const double ang = (double)pos * pow(base, -2.0 * (double)j / (double)(2 * dc));
  double s, c;
  sincos(ang, &s, &c);
  const float cf = (float)c, sf = (float)s;
  q_rot[i] = make_float2(fmaf(qv.x, cf, -qv.y * sf), fmaf(qv.x, sf, qv.y * cf));
  const int64_t at = ((int64_t)h * max_ctx + pos) * dc + j;
  k_cache[at] = make_float2(fmaf(kv.x, cf, -kv.y * sf), fmaf(kv.x, sf, kv.y * cf));
  v_cache[at] = vv;
}

// out = h1 + d, d summed from its partials (and written out).
__global__ void add_sum_kernel(const float2* __restrict__ h1, LayerOut d, int n, float2* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const LayerOut o[1] = {d};
  float2 r[1];
  layer_outs<1, 24>(o, i, r);
  const float2 av = h1[i], bv = r[0];
  out[i] = make_float2(av.x + bv.x, av.y + bv.y);
}

// act = bf16(silu(g) u) per component, g and u summed from their partials
// (and written out).
__global__ void swiglu_sum_kernel(LayerOut g, LayerOut u, int n, uint32_t* __restrict__ act) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const LayerOut o[2] = {g, u};
  float2 r[2];
  layer_outs<2>(o, i, r);
  act[i] = (uint32_t)bf16_rne(silu(r[0].x) * r[1].x) | ((uint32_t)bf16_rne(silu(r[0].y) * r[1].y) << 16);
}

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Plan: header, then the four group tables (q k v; o; gate up; down).
constexpr uint32_t kBlockMagic = 0xFA11B10Cu;
constexpr int kGroups = 4;
struct BlockPlanHeader {
  uint32_t magic, abi;
  int64_t n, n_ff, max_ctx;
  int32_t n_heads, T;
  float eps;
  int32_t fused;  // one-token fp4 groups: the fused path runs
  double rope_base;
  const float* norm_attn;
  const float* norm_mlp;
  // workspace buffers
  uint16_t* z;
  float2 *q, *k, *v, *q_rot;
  float* part;
  uint16_t* o;
  float2 *a, *h1;
  uint16_t* z2;
  float2 *g, *u;
  uint16_t* act;
  float2* d;
  size_t table_off[kGroups];
  size_t table_bytes[kGroups];
};

struct BlockLayout {
  size_t z, q, k, v, q_rot, part, o, a, h1, z2, g, u, act, d, groups[kGroups], total;
};

// the projections of each group call, as indices into desc->codes_*: q k v, o, gate up, down
const int kGroupLayers[kGroups][3] = {{0, 1, 2}, {3, -1, -1}, {4, 5, -1}, {6, -1, -1}};

bool block_desc_ok(const fairy2i_block_desc* d) {
  if (!d || d->n <= 0 || d->n_ff <= 0 || d->n_heads <= 0 || d->max_ctx <= 0) return false;
  if (d->n % d->n_heads != 0 || d->n / d->n_heads > 256 || (d->n / d->n_heads) % 2 != 0) return false;
  if (d->n % 64 != 0 || d->n_ff % 64 != 0) return false;
  if (d->n > (1 << 24) || d->n_ff > (1 << 24) || d->max_ctx > (int64_t)kAttnSlice * kMaxAttnSlices) return false;
  if (d->T < 1 || d->T > FAIRY2I_MAX_STAGES || !(d->eps >= 0.0f) || !(d->rope_base > 0.0)) return false;
  return true;
}

// The group's layer descriptors, pointing at the workspace buffers of `ws`
// (null: a layout pass that only needs the shapes).
int group_layers(const fairy2i_block_desc* d, int gi, char* ws, const BlockLayout& L, fairy2i_wl_layer* out) {
  const int64_t n = d->n, f = d->n_ff;
  int cnt = 0;
  for (int s = 0; s < 3; ++s) {
    const int p = kGroupLayers[gi][s];
    if (p < 0) continue;
    fairy2i_wl_layer l{};
    l.codes_U = d->codes_U[p];
    l.scales_U = d->scales_U[p];
    l.codes_W = d->codes_W[p];
    l.scales_W = d->scales_W[p];
    l.layout = FAIRY2I_LAYOUT_TILED_FP4;
    l.N = (p == 4 || p == 5) ? f : n;
    l.K = (p == 6) ? f : n;
    size_t xoff = 0, yoff = 0;
    switch (p) {
      case 0: xoff = L.z; yoff = L.q; break;
      case 1: xoff = L.z; yoff = L.k; break;
      case 2: xoff = L.z; yoff = L.v; break;
      case 3: xoff = L.o; yoff = L.a; break;
      case 4: xoff = L.z2; yoff = L.g; break;
      case 5: xoff = L.z2; yoff = L.u; break;
      default: xoff = L.act; yoff = L.d; break;
    }
    // placeholders keep the shape checks of the layout pass happy
    l.x = ws ? (const void*)(ws + xoff) : (const void*)d;
    l.y = ws ? reinterpret_cast<float*>(ws + yoff) : reinterpret_cast<float*>(const_cast<fairy2i_block_desc*>(d));
    out[cnt++] = l;
  }
  return cnt;
}

// Workspace layout; the group workspaces need the group shapes only.
bool block_layout(const fairy2i_block_desc* d, BlockLayout& L) {
  const size_t n = (size_t)d->n, f = (size_t)d->n_ff;
  const size_t H = (size_t)d->n_heads, dc = n / H;
  const size_t slices = ((size_t)d->max_ctx + kAttnSlice - 1) / kAttnSlice;
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o += align256(bytes); return at; };
  L.z = take(n * 4);
  L.q = take(n * 8);
  L.k = take(n * 8);
  L.v = take(n * 8);
  L.q_rot = take(n * 8);
  L.part = take(H * slices * (2 + 2 * dc) * 4);
  L.o = take(n * 4);
  L.a = take(n * 8);
  L.h1 = take(n * 8);
  L.z2 = take(n * 4);
  L.g = take(f * 8);
  L.u = take(f * 8);
  L.act = take(f * 4);
  L.d = take(n * 8);
  for (int gi = 0; gi < kGroups; ++gi) {
    fairy2i_wl_layer ls[3];
    const int cnt = group_layers(d, gi, nullptr, L, ls);
    const size_t b = fairy2i_wl_group_workspace_bytes(ls, cnt, d->T, FAIRY2I_ACT_BF16, 1);
    if (b == 0) return false;
    L.groups[gi] = take(b);
  }
  L.total = o;
  return true;
}

inline fairy2i_status hip_st(hipError_t e) { return e == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP; }

void launch_attention(const BlockPlanHeader* hdr, float2* kc, float2* vc, int64_t pos, hipStream_t s) {
  const int n = (int)hdr->n, H = hdr->n_heads, dc = n / H;
  const int64_t n_ctx = pos + 1;
  const int slices = (int)((n_ctx + kAttnSlice - 1) / kAttnSlice);
  const float scale = (float)(1.0 / sqrt((double)(2 * dc)));
  if (dc <= 64)
    hipLaunchKernelGGL(attn_partial_kernel<1>, dim3(slices, H), dim3(kAttnThreads), 0, s, hdr->q_rot, kc, vc, dc, n_ctx,
                       hdr->max_ctx, scale, hdr->part);
  else
    hipLaunchKernelGGL(attn_partial_kernel<4>, dim3(slices, H), dim3(kAttnThreads), 0, s, hdr->q_rot, kc, vc, dc, n_ctx,
                       hdr->max_ctx, scale, hdr->part);
  hipLaunchKernelGGL(attn_combine_kernel, dim3(H), dim3(64), 0, s, hdr->part, slices, dc, hdr->o);
}

// The fused path: the four product launches and eight block kernels.
fairy2i_status block_decode_fused(const void* plan, const void* plan_device, const float2* xin, float2* kc,
                                  float2* vc, int64_t pos, float2* out, hipStream_t s) {
  const auto* hdr = static_cast<const BlockPlanHeader*>(plan);
  const int n = (int)hdr->n, f = (int)hdr->n_ff, dc = n / hdr->n_heads;
  auto gtab = [&](int gi) {
    return reinterpret_cast<const GroupTableHeader*>(static_cast<const char*>(plan) + hdr->table_off[gi]);
  };
  auto layer = [&](int gi, int i) -> const DecLayer& { return reinterpret_cast<const DecLayer*>(gtab(gi) + 1)[i]; };
  auto out_of = [&](int gi, int i) {
    const DecLayer& l = layer(gi, i);
    return LayerOut{l.part, l.y, l.nkc, l.N};
  };
  auto targets = [&](int gi) {
    OperandTargets t{};
    t.count = gtab(gi)->h.n_layers;
    for (int i = 0; i < t.count; ++i) {
      t.xf[i] = layer(gi, i).xf;
      t.xs[i] = layer(gi, i).xs;
    }
    t.nk4 = layer(gi, 0).nk4;
    t.ctr = gtab(gi)->h.coop_ctr;
    return t;
  };
  auto product = [&](int gi) {
    DecLayer none{};
    const auto* td = reinterpret_cast<const DecLayer*>(static_cast<const char*>(plan_device) + hdr->table_off[gi] +
                                                        sizeof(GroupTableHeader));
    launch_f4_product(gtab(gi)->h, none, td, s);
  };
  OperandArgs a{};
  // attention input: RMSNorm of x, operand of q, k, v
  a.K = n;
  a.x = xin;
  a.gamma = hdr->norm_attn;
  a.eps = hdr->eps;
  a.z_out = hdr->z;
  a.t = targets(0);
  launch_operand<kSrcNorm>(a, s);
  product(0);
  hipLaunchKernelGGL(rope_append_sum_kernel, dim3((n + 255) / 256), dim3(256), 0, s, out_of(0, 0), out_of(0, 1),
                     out_of(0, 2), n, dc, pos, hdr->max_ctx, hdr->rope_base, hdr->q_rot, kc, vc);
  launch_attention(hdr, kc, vc, pos, s);
  // output projection input: the attention output as it stands
  a = OperandArgs{};
  a.K = n;
  a.tok = reinterpret_cast<const uint32_t*>(hdr->o);
  a.t = targets(1);
  launch_operand<kSrcBf16>(a, s);
  product(1);
  // MLP input: h1 = x + attention branch, its RMSNorm; operand of gate and up
  a = OperandArgs{};
  a.K = n;
  a.x = xin;
  a.res = out_of(1, 0);
  a.h_out = hdr->h1;
  a.gamma = hdr->norm_mlp;
  a.eps = hdr->eps;
  a.z_out = hdr->z2;
  a.t = targets(2);
  launch_operand<kSrcNorm>(a, s);
  product(2);
  // down projection input: SwiGLU of gate and up
  hipLaunchKernelGGL(swiglu_sum_kernel, dim3((f + 255) / 256), dim3(256), 0, s, out_of(2, 0), out_of(2, 1), f,
                     reinterpret_cast<uint32_t*>(hdr->act));
  a = OperandArgs{};
  a.K = f;
  a.tok = reinterpret_cast<const uint32_t*>(hdr->act);
  a.t = targets(3);
  launch_operand<kSrcBf16>(a, s);
  product(3);
  hipLaunchKernelGGL(add_sum_kernel, dim3((n + 255) / 256), dim3(256), 0, s, hdr->h1, out_of(3, 0), n, out);
  return hip_st(hipGetLastError());
}

}  // namespace

}  // namespace fairy2i

using namespace fairy2i;

extern "C" {

size_t fairy2i_block_workspace_bytes(const fairy2i_block_desc* desc) {
  if (!block_desc_ok(desc)) return 0;
  BlockLayout L;
  return block_layout(desc, L) ? L.total : 0;
}

size_t fairy2i_block_plan_bytes(const fairy2i_block_desc* desc) {
  if (!block_desc_ok(desc)) return 0;
  size_t total = align256(sizeof(BlockPlanHeader));
  for (int gi = 0; gi < kGroups; ++gi) total += align256(fairy2i_wl_group_table_bytes(gi == 0 ? 3 : (gi == 2 ? 2 : 1)));
  return total;
}

fairy2i_status fairy2i_block_build_plan(const fairy2i_block_desc* desc, void* workspace, size_t workspace_bytes,
                                        void* plan, size_t plan_bytes) {
  if (!desc || !workspace || !plan) return FAIRY2I_ERR_NULL;
  if (!block_desc_ok(desc)) return FAIRY2I_ERR_SHAPE;
  for (int p = 0; p < 7; ++p)
    if (!desc->codes_U[p] || !desc->codes_W[p] || !desc->scales_U[p] || !desc->scales_W[p]) return FAIRY2I_ERR_NULL;
  if (!desc->norm_attn || !desc->norm_mlp) return FAIRY2I_ERR_NULL;
  BlockLayout L;
  if (!block_layout(desc, L)) return FAIRY2I_ERR_UNSUPPORTED;
  if (workspace_bytes < L.total) return FAIRY2I_ERR_WORKSPACE;
  if (plan_bytes < fairy2i_block_plan_bytes(desc)) return FAIRY2I_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  char* pl = static_cast<char*>(plan);
  auto* hdr = reinterpret_cast<BlockPlanHeader*>(pl);
  memset(hdr, 0, sizeof(BlockPlanHeader));
  hdr->magic = kBlockMagic;
  hdr->abi = (uint32_t)fairy2i_abi_version();
  hdr->n = desc->n;
  hdr->n_ff = desc->n_ff;
  hdr->max_ctx = desc->max_ctx;
  hdr->n_heads = desc->n_heads;
  hdr->T = desc->T;
  hdr->eps = desc->eps;
  hdr->rope_base = desc->rope_base;
  hdr->norm_attn = desc->norm_attn;
  hdr->norm_mlp = desc->norm_mlp;
  hdr->z = reinterpret_cast<uint16_t*>(ws + L.z);
  hdr->q = reinterpret_cast<float2*>(ws + L.q);
  hdr->k = reinterpret_cast<float2*>(ws + L.k);
  hdr->v = reinterpret_cast<float2*>(ws + L.v);
  hdr->q_rot = reinterpret_cast<float2*>(ws + L.q_rot);
  hdr->part = reinterpret_cast<float*>(ws + L.part);
  hdr->o = reinterpret_cast<uint16_t*>(ws + L.o);
  hdr->a = reinterpret_cast<float2*>(ws + L.a);
  hdr->h1 = reinterpret_cast<float2*>(ws + L.h1);
  hdr->z2 = reinterpret_cast<uint16_t*>(ws + L.z2);
  hdr->g = reinterpret_cast<float2*>(ws + L.g);
  hdr->u = reinterpret_cast<float2*>(ws + L.u);
  hdr->act = reinterpret_cast<uint16_t*>(ws + L.act);
  hdr->d = reinterpret_cast<float2*>(ws + L.d);
  size_t off = align256(sizeof(BlockPlanHeader));
  for (int gi = 0; gi < kGroups; ++gi) {
    fairy2i_wl_layer ls[3];
    const int cnt = group_layers(desc, gi, ws, L, ls);
    const size_t tb = fairy2i_wl_group_table_bytes(cnt);
    const size_t gws = fairy2i_wl_group_workspace_bytes(ls, cnt, desc->T, FAIRY2I_ACT_BF16, 1);
    const fairy2i_status st = fairy2i_wl_group_build_table(ls, cnt, desc->T, FAIRY2I_ACT_BF16, 1, ws + L.groups[gi],
                                                           gws, pl + off, tb);
    if (st != FAIRY2I_OK) return st;
    hdr->table_off[gi] = off;
    hdr->table_bytes[gi] = tb;
    off += align256(tb);
  }
  hdr->fused = desc->n <= kOpMaxK && desc->n_ff <= kOpMaxK;
  for (int gi = 0; gi < kGroups; ++gi) {
    const DecHeader& h = reinterpret_cast<const GroupTableHeader*>(pl + hdr->table_off[gi])->h;
    if (h.mode != kModeBf16F4 || h.B != 1 || h.bands != 2 || h.nc != 8 || h.ntile != 1) hdr->fused = 0;
  }
  return FAIRY2I_OK;
}

fairy2i_status fairy2i_block_intermediates(const void* plan, void** ptrs) {
  if (!plan || !ptrs) return FAIRY2I_ERR_NULL;
  const auto* hdr = static_cast<const BlockPlanHeader*>(plan);
  if (hdr->magic != kBlockMagic || hdr->abi != (uint32_t)fairy2i_abi_version()) return FAIRY2I_ERR_UNSUPPORTED;
  void* const p[12] = {hdr->z, hdr->q_rot, hdr->v, hdr->o, hdr->a, hdr->h1,
                       hdr->z2, hdr->g, hdr->u, hdr->act, hdr->d, hdr->k};
  for (int i = 0; i < 12; ++i) ptrs[i] = p[i];
  return FAIRY2I_OK;
}

fairy2i_status fairy2i_block_decode(const void* plan, const void* plan_device, const float* x, float* k_cache,
                                    float* v_cache, int64_t pos, float* out, void* stream) {
  if (!plan || !plan_device || !x || !k_cache || !v_cache || !out) return FAIRY2I_ERR_NULL;
  const auto* hdr = static_cast<const BlockPlanHeader*>(plan);
  if (hdr->magic != kBlockMagic || hdr->abi != (uint32_t)fairy2i_abi_version()) return FAIRY2I_ERR_UNSUPPORTED;
  if (pos < 0 || pos >= hdr->max_ctx) return FAIRY2I_ERR_SHAPE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n = (int)hdr->n, f = (int)hdr->n_ff, H = hdr->n_heads, dc = n / H;
  const int64_t n_ctx = pos + 1;
  const int slices = (int)((n_ctx + kAttnSlice - 1) / kAttnSlice);
  auto group = [&](int gi) -> fairy2i_status {
    return fairy2i_wl_matmul_group(static_cast<const char*>(plan) + hdr->table_off[gi],
                                   static_cast<const char*>(plan_device) + hdr->table_off[gi], stream);
  };
  const float2* xin = reinterpret_cast<const float2*>(x);
  float2* kc = reinterpret_cast<float2*>(k_cache);
  float2* vc = reinterpret_cast<float2*>(v_cache);
  hipError_t e;
  fairy2i_status st;
  const float scale = (float)(1.0 / sqrt((double)(2 * dc)));
  if (hdr->fused) return block_decode_fused(plan, plan_device, xin, kc, vc, pos, reinterpret_cast<float2*>(out), s);
  hipLaunchKernelGGL(add_rmsnorm_kernel, dim3(1), dim3(kNormThreads), 0, s, xin, nullptr, nullptr, hdr->norm_attn,
                     hdr->eps, n, hdr->z);
  if ((e = hipGetLastError()) != hipSuccess) return hip_st(e);
  if ((st = group(0)) != FAIRY2I_OK) return st;
  hipLaunchKernelGGL(rope_append_kernel, dim3((n + 255) / 256), dim3(256), 0, s, hdr->q, hdr->k, hdr->v, n, dc, pos,
                     hdr->max_ctx, hdr->rope_base, hdr->q_rot, kc, vc);
  if (dc <= 64)
    hipLaunchKernelGGL(attn_partial_kernel<1>, dim3(slices, H), dim3(kAttnThreads), 0, s, hdr->q_rot, kc, vc, dc, n_ctx,
                       hdr->max_ctx, scale, hdr->part);
  else
    hipLaunchKernelGGL(attn_partial_kernel<4>, dim3(slices, H), dim3(kAttnThreads), 0, s, hdr->q_rot, kc, vc, dc, n_ctx,
                       hdr->max_ctx, scale, hdr->part);
  hipLaunchKernelGGL(attn_combine_kernel, dim3(H), dim3(64), 0, s, hdr->part, slices, dc, hdr->o);
  if ((e = hipGetLastError()) != hipSuccess) return hip_st(e);
  if ((st = group(1)) != FAIRY2I_OK) return st;
  hipLaunchKernelGGL(add_rmsnorm_kernel, dim3(1), dim3(kNormThreads), 0, s, xin, hdr->a, hdr->h1, hdr->norm_mlp,
                     hdr->eps, n, hdr->z2);
  if ((e = hipGetLastError()) != hipSuccess) return hip_st(e);
  if ((st = group(2)) != FAIRY2I_OK) return st;
  hipLaunchKernelGGL(swiglu_kernel, dim3((f + 255) / 256), dim3(256), 0, s, hdr->g, hdr->u, f, hdr->act);
  if ((e = hipGetLastError()) != hipSuccess) return hip_st(e);
  if ((st = group(3)) != FAIRY2I_OK) return st;
  hipLaunchKernelGGL(add_kernel, dim3((n + 255) / 256), dim3(256), 0, s, hdr->h1, hdr->d, n,
                     reinterpret_cast<float2*>(out));
  return hip_st(hipGetLastError());
}

}  // extern "C"
