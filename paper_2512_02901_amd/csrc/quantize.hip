// Recursive residual PhaseQuant of one complex matrix (Sec. 3.3 formal
// definition, with the projection, axis scales and dequantisation of
// Sec. 3.2).
//
// A fill kernel clears the per-stage totals; then stage t runs two kernels on
// the caller's stream:
//   qz_stage_kernel    one thread per packed byte (4 consecutive entries of a
//                      row): rebuilds the float64 residual from M and the
//                      codes/scales of stages < t, projects it, writes the
//                      byte of stage-t codes, and adds |Re r| (k even) or
//                      |Im r| (k odd) into an exact fixed-point sum (a
//                      window of limbs in registers per thread, the rest in
//                      LDS).  Each block then adds its accumulator words into
//                      one of 16 copies of the stage total with 64-bit
//                      integer atomics (exact, so the total does not depend
//                      on the order blocks arrive in).
//   qz_finalize_kernel rounds each exact mean once to float32 -> scales[t].
// Stage t+1 reads scales[t] from device memory; nothing returns to the host.
#include "common.h"
#include "superacc.h"

namespace fairy2i {

namespace {

constexpr int kPartWords = 2 * SA_LIMBS + 2;  // acc[2][SA_LIMBS], cnt[2]

// Eq. (ifairy-proj) by exact comparisons (floor-form ties, 0 -> +1).
__device__ inline uint32_t project_code(double a, double b) {
  if (b > 0.0 && -b < a && a <= b) return 1u;
  if (a < 0.0 && a < b && b <= -a) return 2u;
  if (b < 0.0 && b <= a && a < -b) return 3u;
  return 0u;
}

// A thread's share of an exact sum: kSaWin limbs of 64 bits from limb w0 on
// (w0 < 0: not yet placed), in registers.  A value's three 32-bit chunks go
// to limbs limb .. limb + 2 of the window when they fit (w0 is set one limb
// below the first value's, so values within about 2^32 of it, the usual
// spread of a weight matrix, fit), else straight to the block's LDS
// accumulator.  Either way the integer total is the same.
constexpr int kSaWin = 5;
struct SaWin {
  unsigned long long w[kSaWin];
  int w0;
};

__device__ inline void sa_win_init(SaWin& s) {
#pragma unroll
  for (int j = 0; j < kSaWin; ++j) s.w[j] = 0ull;
  s.w0 = -1;
}

__device__ inline void sa_add(SaWin& s, unsigned long long* acc, double v) {
  if (v == 0.0) return;
  int limb;
  uint32_t lo, mid, hi;
  sa_split(v, &limb, &lo, &mid, &hi);
  if (s.w0 < 0) s.w0 = limb > 0 ? limb - 1 : 0;
  const int d = limb - s.w0;
  if (d >= 0 && d + 2 < kSaWin) {
#pragma unroll
    for (int j = 0; j < kSaWin; ++j)
      s.w[j] += (unsigned long long)(j == d ? lo : (j == d + 1 ? mid : (j == d + 2 ? hi : 0u)));
    return;
  }
  if (lo) atomicAdd(&acc[limb], (unsigned long long)lo);
  if (mid) atomicAdd(&acc[limb + 1], (unsigned long long)mid);
  if (hi) atomicAdd(&acc[limb + 2], (unsigned long long)hi);
}

// The window's limbs into the block's accumulator (a nonzero limb w0 + j
// holds chunks of values whose limbs lie inside the accumulator).
__device__ inline void sa_flush(const SaWin& s, unsigned long long* acc) {
#pragma unroll
  for (int j = 0; j < kSaWin; ++j)
    if (s.w[j] && s.w0 + j < SA_LIMBS) atomicAdd(&acc[s.w0 + j], s.w[j]);
}

// Rebuild the float64 residual of one entry from M and the codes/scales of
// stages < t (R(tp+1) = R(tp) - W^(tp)), project it, and add its magnitude
// on the chosen axis to the thread's exact partial sums.  Returns the code.
__device__ inline uint32_t qz_entry(float2 m, const uint32_t* prev, int e, int t, const double* s_re,
                                    const double* s_im, unsigned long long (*acc)[SA_LIMBS], SaWin (&win)[2],
                                    unsigned long long& n_re, unsigned long long& n_im) {
  double re = (double)m.x, im = (double)m.y;
#pragma unroll
  for (int tp = 0; tp < FAIRY2I_MAX_STAGES; ++tp) {
    if (tp >= t) break;
    const uint32_t k = (prev[tp] >> (2 * e)) & 3u;
    if (k == 0u) re = re - s_re[tp];
    else if (k == 2u) re = re + s_re[tp];
    else if (k == 1u) im = im - s_im[tp];
    else im = im + s_im[tp];
  }
  const uint32_t k = project_code(re, im);
  // (counts by arithmetic: a branch on which counter to bump lets the
  // compiler turn the pair into an indexed array in scratch)
  const unsigned long long odd = k & 1u;
  n_im += odd;
  n_re += 1ull - odd;
  if (odd) sa_add(win[1], acc[1], fabs(im));
  else sa_add(win[0], acc[0], fabs(re));
  return k;
}

// Copies of a stage's total: block b adds into copy b % kTotCopies, so each
// total word takes 1/kTotCopies of the blocks' atomics; the finalize kernel
// adds the copies (integers: the order does not matter).
constexpr int kTotCopies = 16;
constexpr int kQzUnroll = 4;  // bytes a thread loads before it quantises them

__global__ __launch_bounds__(kQzThreads) void qz_stage_kernel(
    const float2* __restrict__ M, int64_t nbytes, uint8_t* __restrict__ codes,
    const float* __restrict__ scales, int t, unsigned long long* __restrict__ tot) {
  __shared__ unsigned long long acc[2][SA_LIMBS];
  __shared__ unsigned long long cnt[2];
  for (int i = threadIdx.x; i < 2 * SA_LIMBS; i += blockDim.x) (&acc[0][0])[i] = 0ull;
  if (threadIdx.x < 2) cnt[threadIdx.x] = 0ull;
  __syncthreads();

  double s_re[FAIRY2I_MAX_STAGES], s_im[FAIRY2I_MAX_STAGES];
#pragma unroll
  for (int tp = 0; tp < FAIRY2I_MAX_STAGES; ++tp) {
    s_re[tp] = tp < t ? (double)scales[2 * tp] : 0.0;
    s_im[tp] = tp < t ? (double)scales[2 * tp + 1] : 0.0;
  }
  unsigned long long n_re = 0, n_im = 0;
  SaWin win[2];
  sa_win_init(win[0]);
  sa_win_init(win[1]);
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const bool al16 = (reinterpret_cast<uintptr_t>(M) & 15) == 0;  // a byte's 4 entries as two 16-byte loads
  for (int64_t b0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b0 < nbytes; b0 += kQzUnroll * stride) {
    // the loads of kQzUnroll bytes (entries and earlier codes) first
    float4 mv[kQzUnroll][2];
    uint32_t prev[kQzUnroll][FAIRY2I_MAX_STAGES];
#pragma unroll
    for (int u = 0; u < kQzUnroll; ++u) {
      const int64_t bi = b0 + u * stride;
      const bool ok = bi < nbytes;
      mv[u][0] = mv[u][1] = make_float4(0.f, 0.f, 0.f, 0.f);
      if (ok && al16) {
        const float4* m4 = reinterpret_cast<const float4*>(M + 4 * bi);
        mv[u][0] = m4[0];
        mv[u][1] = m4[1];
      } else if (ok) {
        const float2 a0 = M[4 * bi], a1 = M[4 * bi + 1], a2 = M[4 * bi + 2], a3 = M[4 * bi + 3];
        mv[u][0] = make_float4(a0.x, a0.y, a1.x, a1.y);
        mv[u][1] = make_float4(a2.x, a2.y, a3.x, a3.y);
      }
#pragma unroll
      for (int tp = 0; tp < FAIRY2I_MAX_STAGES; ++tp) prev[u][tp] = (ok && tp < t) ? codes[(int64_t)tp * nbytes + bi] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kQzUnroll; ++u) {
      const int64_t bi = b0 + u * stride;
      if (bi >= nbytes) break;
      const float2 m[4] = {make_float2(mv[u][0].x, mv[u][0].y), make_float2(mv[u][0].z, mv[u][0].w),
                           make_float2(mv[u][1].x, mv[u][1].y), make_float2(mv[u][1].z, mv[u][1].w)};
      uint32_t out = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        out |= qz_entry(m[e], prev[u], e, t, s_re, s_im, acc, win, n_re, n_im) << (2 * e);
      codes[(int64_t)t * nbytes + bi] = (uint8_t)out;
    }
  }
  sa_flush(win[0], acc[0]);
  sa_flush(win[1], acc[1]);
  if (n_re) atomicAdd(&cnt[0], n_re);
  if (n_im) atomicAdd(&cnt[1], n_im);
  __syncthreads();
  // the block's words into its copy of the stage total: 64-bit integer
  // additions, exact and independent of the order in which blocks arrive
  unsigned long long* tc = tot + (int64_t)(blockIdx.x % kTotCopies) * kPartWords;
  for (int i = threadIdx.x; i < kPartWords; i += blockDim.x) {
    const unsigned long long v = i < 2 * SA_LIMBS ? (&acc[0][0])[i] : cnt[i - 2 * SA_LIMBS];
    if (v) atomicAdd(&tc[i], v);
  }
}

// The stage's totals are read into LDS by all lanes at once (one round of
// loads, not one per limb of the carry chain), then rounded.
__global__ __launch_bounds__(kPartWords) void qz_finalize_kernel(const unsigned long long* __restrict__ tot,
                                                                 float* __restrict__ scales_t) {
  __shared__ uint64_t w[kPartWords];
  {
    const int i = threadIdx.x;  // one word of the total per thread, the copies' loads in flight together
    uint64_t c[kTotCopies];
#pragma unroll
    for (int k = 0; k < kTotCopies; ++k) c[k] = tot[(int64_t)k * kPartWords + i];
    uint64_t v = 0;
#pragma unroll
    for (int k = 0; k < kTotCopies; ++k) v += c[k];
    w[i] = v;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    const uint64_t n = w[2 * SA_LIMBS + threadIdx.x];
    scales_t[threadIdx.x] = n ? sa_mean_to_f32(w + threadIdx.x * SA_LIMBS, n) : 0.0f;
  }
}

// Per-group scales: one block per (row, group of G columns).  The block
// quantises the group's entries at stage t exactly as qz_stage_kernel does,
// with the residual rebuilt from the group's own scales of earlier stages,
// and rounds the group's two exact means once to float32 into
// scales[t][row][g][axis].  No cross-block reduction is needed.
constexpr int kQzgThreads = 64;

__global__ __launch_bounds__(kQzgThreads) void qzg_stage_kernel(const float2* __restrict__ M, int64_t N, int64_t K,
                                                                 int64_t G, int64_t ngroups,
                                                                 uint8_t* __restrict__ codes,
                                                                 float* __restrict__ scales, int t) {
  __shared__ unsigned long long acc[2][SA_LIMBS];
  __shared__ unsigned long long cnt[2];
  for (int i = threadIdx.x; i < 2 * SA_LIMBS; i += blockDim.x) (&acc[0][0])[i] = 0ull;
  if (threadIdx.x < 2) cnt[threadIdx.x] = 0ull;
  __syncthreads();
  const int64_t row = (int64_t)blockIdx.x / ngroups;
  const int64_t g = (int64_t)blockIdx.x - row * ngroups;
  const int64_t j0 = g * G, j1 = j0 + G < K ? j0 + G : K;  // columns of the group (multiples of 4)
  const int64_t nbytes = N * K / 4;
  double s_re[FAIRY2I_MAX_STAGES], s_im[FAIRY2I_MAX_STAGES];
#pragma unroll
  for (int tp = 0; tp < FAIRY2I_MAX_STAGES; ++tp) {
    const float* sp = scales + ((tp * N + row) * ngroups + g) * 2;
    s_re[tp] = tp < t ? (double)sp[0] : 0.0;
    s_im[tp] = tp < t ? (double)sp[1] : 0.0;
  }
  unsigned long long n_re = 0, n_im = 0;
  SaWin win[2];
  sa_win_init(win[0]);
  sa_win_init(win[1]);
  for (int64_t bi = row * (K / 4) + j0 / 4 + threadIdx.x; bi < row * (K / 4) + j1 / 4; bi += blockDim.x) {
    uint32_t prev[FAIRY2I_MAX_STAGES];
#pragma unroll
    for (int tp = 0; tp < FAIRY2I_MAX_STAGES; ++tp) prev[tp] = tp < t ? codes[(int64_t)tp * nbytes + bi] : 0u;
    uint32_t out = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      out |= qz_entry(M[4 * bi + e], prev, e, t, s_re, s_im, acc, win, n_re, n_im) << (2 * e);
    codes[(int64_t)t * nbytes + bi] = (uint8_t)out;
  }
  sa_flush(win[0], acc[0]);
  sa_flush(win[1], acc[1]);
  if (n_re) atomicAdd(&cnt[0], n_re);
  if (n_im) atomicAdd(&cnt[1], n_im);
  __syncthreads();
  if (threadIdx.x < 2) {
    const unsigned long long n = cnt[threadIdx.x];
    scales[((t * N + row) * ngroups + g) * 2 + threadIdx.x] =
        n ? sa_mean_to_f32(reinterpret_cast<const uint64_t*>(acc[threadIdx.x]), n) : 0.0f;
  }
}

__global__ __launch_bounds__(256) void qz_zero_kernel(unsigned long long* __restrict__ p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0ull;
}

int quantize_blocks(int64_t N, int64_t K) {
  const int64_t nbytes = N * K / 4;
  int64_t b = (nbytes + kQzThreads - 1) / kQzThreads;
  if (b > kQzMaxBlocks) b = kQzMaxBlocks;
  if (b < 1) b = 1;
  return (int)b;
}

}  // namespace

hipError_t launch_quantize_grouped(const float2* M, int64_t N, int64_t K, int T, int64_t G, uint8_t* codes,
                                   float* scales, hipStream_t stream) {
  const int64_t ngroups = (K + G - 1) / G;
  for (int t = 0; t < T; ++t) {
    hipLaunchKernelGGL(qzg_stage_kernel, dim3((unsigned)(N * ngroups)), dim3(kQzgThreads), 0, stream, M, N, K, G,
                       ngroups, codes, scales, t);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

size_t quantize_workspace_bytes(int64_t N, int64_t K) {
  (void)N;
  (void)K;
  return (size_t)FAIRY2I_MAX_STAGES * kTotCopies * kPartWords * sizeof(unsigned long long);  // totals per stage
}

hipError_t launch_quantize(const float2* M, int64_t N, int64_t K, int T, uint8_t* codes,
                           float* scales, void* workspace, hipStream_t stream) {
  const int nblk = quantize_blocks(N, K);
  const int64_t nbytes = N * K / 4;
  auto* tot = static_cast<unsigned long long*>(workspace);
  hipLaunchKernelGGL(qz_zero_kernel, dim3(1), dim3(256), 0, stream, tot, T * kTotCopies * kPartWords);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  for (int t = 0; t < T; ++t) {
    unsigned long long* tot_t = tot + (int64_t)t * kTotCopies * kPartWords;
    hipLaunchKernelGGL(qz_stage_kernel, dim3(nblk), dim3(kQzThreads), 0, stream, M, nbytes, codes,
                       scales, t, tot_t);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(qz_finalize_kernel, dim3(1), dim3(kPartWords), 0, stream, tot_t, scales + 2 * t);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace fairy2i
