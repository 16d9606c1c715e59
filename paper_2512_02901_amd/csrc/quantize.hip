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
//                      |Im r| (k odd) into an exact fixed-point accumulator
//                      in LDS.  Each block then adds its accumulator words into the
//                      stage total with 64-bit integer atomics (exact, so the
//                      total does not depend on the order blocks arrive in).
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

__device__ inline void sa_add_lds(unsigned long long* acc, double v) {
  if (v == 0.0) return;
  int limb;
  uint32_t lo, mid, hi;
  sa_split(v, &limb, &lo, &mid, &hi);
  if (lo) atomicAdd(&acc[limb], (unsigned long long)lo);
  if (mid) atomicAdd(&acc[limb + 1], (unsigned long long)mid);
  if (hi) atomicAdd(&acc[limb + 2], (unsigned long long)hi);
}

// Rebuild the float64 residual of one entry from M and the codes/scales of
// stages < t (R(tp+1) = R(tp) - W^(tp)), project it, and add its magnitude
// on the chosen axis to the block's exact accumulator.  Returns the code.
__device__ inline uint32_t qz_entry(float2 m, const uint32_t* prev, int e, int t, const double* s_re,
                                    const double* s_im, unsigned long long (*acc)[SA_LIMBS],
                                    unsigned long long& n_re, unsigned long long& n_im) {
  double re = (double)m.x, im = (double)m.y;
  for (int tp = 0; tp < t; ++tp) {
    const uint32_t k = (prev[tp] >> (2 * e)) & 3u;
    if (k == 0u) re = re - s_re[tp];
    else if (k == 2u) re = re + s_re[tp];
    else if (k == 1u) im = im - s_im[tp];
    else im = im + s_im[tp];
  }
  const uint32_t k = project_code(re, im);
  if (k & 1u) {
    sa_add_lds(acc[1], fabs(im));
    ++n_im;
  } else {
    sa_add_lds(acc[0], fabs(re));
    ++n_re;
  }
  return k;
}

__global__ __launch_bounds__(kQzThreads) void qz_stage_kernel(
    const float2* __restrict__ M, int64_t nbytes, uint8_t* __restrict__ codes,
    const float* __restrict__ scales, int t, unsigned long long* __restrict__ tot) {
  __shared__ unsigned long long acc[2][SA_LIMBS];
  __shared__ unsigned long long cnt[2];
  for (int i = threadIdx.x; i < 2 * SA_LIMBS; i += blockDim.x) (&acc[0][0])[i] = 0ull;
  if (threadIdx.x < 2) cnt[threadIdx.x] = 0ull;
  __syncthreads();

  double s_re[FAIRY2I_MAX_STAGES], s_im[FAIRY2I_MAX_STAGES];
  for (int tp = 0; tp < t; ++tp) {
    s_re[tp] = (double)scales[2 * tp];
    s_im[tp] = (double)scales[2 * tp + 1];
  }
  unsigned long long n_re = 0, n_im = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t bi = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; bi < nbytes; bi += stride) {
    uint32_t prev[FAIRY2I_MAX_STAGES];
    for (int tp = 0; tp < t; ++tp) prev[tp] = codes[(int64_t)tp * nbytes + bi];
    uint32_t out = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) out |= qz_entry(M[4 * bi + e], prev, e, t, s_re, s_im, acc, n_re, n_im) << (2 * e);
    codes[(int64_t)t * nbytes + bi] = (uint8_t)out;
  }
  if (n_re) atomicAdd(&cnt[0], n_re);
  if (n_im) atomicAdd(&cnt[1], n_im);
  __syncthreads();
  // the block's words into the stage total: 64-bit integer additions, exact
  // and independent of the order in which blocks arrive
  for (int i = threadIdx.x; i < kPartWords; i += blockDim.x) {
    const unsigned long long v = i < 2 * SA_LIMBS ? (&acc[0][0])[i] : cnt[i - 2 * SA_LIMBS];
    if (v) atomicAdd(&tot[i], v);
  }
}

__global__ __launch_bounds__(64) void qz_finalize_kernel(const unsigned long long* __restrict__ tot,
                                                         float* __restrict__ scales_t) {
  if (threadIdx.x < 2) {
    const unsigned long long n = tot[2 * SA_LIMBS + threadIdx.x];
    scales_t[threadIdx.x] =
        n ? sa_mean_to_f32(reinterpret_cast<const uint64_t*>(tot + threadIdx.x * SA_LIMBS), n) : 0.0f;
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
  for (int tp = 0; tp < t; ++tp) {
    const float* sp = scales + ((tp * N + row) * ngroups + g) * 2;
    s_re[tp] = (double)sp[0];
    s_im[tp] = (double)sp[1];
  }
  unsigned long long n_re = 0, n_im = 0;
  for (int64_t bi = row * (K / 4) + j0 / 4 + threadIdx.x; bi < row * (K / 4) + j1 / 4; bi += blockDim.x) {
    uint32_t prev[FAIRY2I_MAX_STAGES];
    for (int tp = 0; tp < t; ++tp) prev[tp] = codes[(int64_t)tp * nbytes + bi];
    uint32_t out = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) out |= qz_entry(M[4 * bi + e], prev, e, t, s_re, s_im, acc, n_re, n_im) << (2 * e);
    codes[(int64_t)t * nbytes + bi] = (uint8_t)out;
  }
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
  return (size_t)FAIRY2I_MAX_STAGES * kPartWords * sizeof(unsigned long long);  // one total per stage
}

hipError_t launch_quantize(const float2* M, int64_t N, int64_t K, int T, uint8_t* codes,
                           float* scales, void* workspace, hipStream_t stream) {
  const int nblk = quantize_blocks(N, K);
  const int64_t nbytes = N * K / 4;
  auto* tot = static_cast<unsigned long long*>(workspace);
  hipLaunchKernelGGL(qz_zero_kernel, dim3(1), dim3(256), 0, stream, tot, T * kPartWords);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  for (int t = 0; t < T; ++t) {
    unsigned long long* tot_t = tot + (int64_t)t * kPartWords;
    hipLaunchKernelGGL(qz_stage_kernel, dim3(nblk), dim3(kQzThreads), 0, stream, M, nbytes, codes,
                       scales, t, tot_t);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(qz_finalize_kernel, dim3(1), dim3(64), 0, stream, tot_t, scales + 2 * t);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace fairy2i
