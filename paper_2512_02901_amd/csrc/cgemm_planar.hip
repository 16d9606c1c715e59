// Complex GEMM with Gauss's three real products (Sec. 3.2, remark (iii)) in
// planar form: the product itself is three plain real GEMMs,
//     P1 = Ar Br^T,   P2 = Ai Bi^T,   P3 = (Ar + Ai)(Br + Bi)^T,
// so they run as one batched bf16 GEMM of the vendor library (hipBLASLt,
// float32 accumulation), between two kernels of this file:
//   gauss_planes_kernel   an operand (either layout, float32 or bf16 pairs,
//                         conjugated or not, one or two K segments) into
//                         three bf16 planes [3][rows][Kp], K contiguous:
//                         Re, Im and Re + Im (the sum formed in float32 from
//                         the inputs and rounded once, nearest-even)
//   gauss_combine_kernel  C (+)= (P1 - P2) + i (P3 - P1 - P2)
// The planes round exactly as the single-kernel fairy2i_cgemm_gauss does;
// only the order of the float32 accumulation inside the products differs.
#include "common.h"

#include <hipblaslt/hipblaslt.h>

#include <map>
#include <mutex>
#include <tuple>

namespace fairy2i {

namespace {

constexpr int kPlaneTile = 64;          // rows x k per block of the plane kernel
constexpr int64_t kPlaneKAlign = 64;    // plane rows padded to a multiple of 64 values (128 bytes)
constexpr size_t kLtWorkspaceBytes = (size_t)32 << 20;

inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

__device__ inline uint16_t bf16_nearest_even(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

struct PlaneOp {
  const void* p;
  int64_t ld;
  int32_t dtype, trans, conj, pad_;
};

// One complex value of an operand (zero outside the segment).
__device__ inline float2 op_value(const PlaneOp& op, int64_t idx) {
  if (op.dtype == FAIRY2I_ACT_BF16) {
    const uint32_t w = static_cast<const uint32_t*>(op.p)[idx];
    return make_float2(__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u));
  }
  return static_cast<const float2*>(op.p)[idx];
}

// Block (blockIdx.y, blockIdx.x): rows r0 .. r0 + 63 and segment columns
// k0 .. k0 + 63 of one segment of `rows` x Ks values, written to plane
// columns koff + k; columns at or past Ks (up to the launch's width: the
// padding after the last segment) are written as zeros.
__global__ __launch_bounds__(256) void gauss_planes_kernel(PlaneOp op, int64_t rows, int64_t Ks, int64_t koff,
                                                           int64_t width, int64_t Kp, uint16_t* __restrict__ planes) {
  __shared__ uint16_t tile[3][kPlaneTile][kPlaneTile + 8];
  const int t = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.y * kPlaneTile, k0 = (int64_t)blockIdx.x * kPlaneTile;
  // load 16 consecutive values along the operand's contiguous dimension
  const int a = t >> 2, b = (t & 3) * 16;  // (row, k run) or (k, row run)
#pragma unroll 4
  for (int e = 0; e < 16; ++e) {
    const int64_t r = op.trans ? r0 + b + e : r0 + a;
    const int64_t k = op.trans ? k0 + a : k0 + b + e;
    float2 v = make_float2(0.0f, 0.0f);
    if (r < rows && k < Ks) v = op_value(op, op.trans ? k * op.ld + r : r * op.ld + k);
    if (op.conj) v.y = -v.y;
    const int lr = op.trans ? b + e : a, lk = op.trans ? a : b + e;
    tile[0][lr][lk] = bf16_nearest_even(v.x);
    tile[1][lr][lk] = bf16_nearest_even(v.y);
    tile[2][lr][lk] = bf16_nearest_even(v.x + v.y);
  }
  __syncthreads();
  // store: thread (row a, 16 columns from b) of each plane
  const int64_t r = r0 + a;
  if (r >= rows) return;
  const int64_t kc = k0 + b;  // first segment column of this thread
  const int64_t nk = width - kc < 16 ? width - kc : 16;
  if (nk <= 0) return;
#pragma unroll
  for (int pl = 0; pl < 3; ++pl) {
    uint16_t* dst = planes + ((int64_t)pl * rows + r) * Kp + koff + kc;
    if (nk == 16 && (reinterpret_cast<uintptr_t>(dst) & 15) == 0) {
      const uint4* src = reinterpret_cast<const uint4*>(&tile[pl][a][b]);
      reinterpret_cast<uint4*>(dst)[0] = src[0];
      reinterpret_cast<uint4*>(dst)[1] = src[1];
    } else {
      for (int e = 0; e < nk; ++e) dst[e] = tile[pl][a][b + e];
    }
  }
}

// C[m][n] (+)= (P1 - P2) + i (P3 - P1 - P2), P = [3][M][N] float32; blocks
// walk rows (y) and 256-column runs (x).
__global__ __launch_bounds__(256) void gauss_combine_kernel(const float* __restrict__ P, int64_t M, int64_t N,
                                                            float2* __restrict__ C, int64_t ldc, int accumulate) {
  const int64_t MN = M * N;
  for (int64_t m = blockIdx.y; m < M; m += gridDim.y)
    for (int64_t n = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; n < N; n += (int64_t)gridDim.x * blockDim.x) {
      const int64_t i = m * N + n;
      const float p1 = P[i], p2 = P[MN + i], p3 = P[2 * MN + i];
      const float re = p1 - p2;
      const float im = (p3 - p1) - p2;
      float2* c = C + m * ldc + n;
      if (accumulate) {
        const float2 o = *c;
        *c = make_float2(o.x + re, o.y + im);
      } else {
        *c = make_float2(re, im);
      }
    }
}

// ------------------------------------------------------------ hipBLASLt ---
// One handle per device, created on first use; the chosen algorithm per
// problem shape is kept, so a shape pays for the library's heuristic once.
std::mutex g_lt_mutex;
std::map<int, hipblasLtHandle_t> g_lt_handles;
std::map<std::tuple<int, int64_t, int64_t, int64_t>, hipblasLtMatmulAlgo_t> g_lt_algos;

struct LtDescs {
  hipblasLtMatmulDesc_t op = nullptr;
  hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
  ~LtDescs() {
    if (a) hipblasLtMatrixLayoutDestroy(a);
    if (b) hipblasLtMatrixLayoutDestroy(b);
    if (c) hipblasLtMatrixLayoutDestroy(c);
    if (op) hipblasLtMatmulDescDestroy(op);
  }
};

bool lt_ok(hipblasStatus_t s) { return s == HIPBLAS_STATUS_SUCCESS; }

// P[z] (row-major M x N) = Aplanes[z] (M x Kp) Bplanes[z] (N x Kp)^T for z < 3.
// Column-major view: P[z]^T (N x M, ld N) = Bplanes[z]^T (op T of a Kp x N
// matrix, ld Kp) times Aplanes[z]^T (a Kp x M matrix, ld Kp).
// The current device's handle (created on first use) in *h.
fairy2i_status lt_handle(int* dev, hipblasLtHandle_t* h) {
  if (hipGetDevice(dev) != hipSuccess) return FAIRY2I_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_lt_mutex);
  auto it = g_lt_handles.find(*dev);
  if (it == g_lt_handles.end()) {
    if (!lt_ok(hipblasLtCreate(h))) return FAIRY2I_ERR_HIP;
    g_lt_handles[*dev] = *h;
  } else {
    *h = it->second;
  }
  return FAIRY2I_OK;
}

// The library's first heuristic choice for a problem, or false.
bool lt_pick(hipblasLtHandle_t h, const LtDescs& d, hipblasLtMatmulAlgo_t* algo) {
  hipblasLtMatmulPreference_t pref = nullptr;
  const uint64_t wsb = kLtWorkspaceBytes;
  hipblasLtMatmulHeuristicResult_t res[1];
  int found = 0;
  const bool ok =
      lt_ok(hipblasLtMatmulPreferenceCreate(&pref)) &&
      lt_ok(hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsb, sizeof(wsb))) &&
      lt_ok(hipblasLtMatmulAlgoGetHeuristic(h, d.op, d.a, d.b, d.c, d.c, pref, 1, res, &found));
  if (pref) hipblasLtMatmulPreferenceDestroy(pref);
  if (!ok || found < 1 || res[0].workspaceSize > kLtWorkspaceBytes) return false;
  *algo = res[0].algo;
  return true;
}

fairy2i_status lt_products(const uint16_t* Ap, const uint16_t* Bp, float* P, int64_t M, int64_t N, int64_t Kp,
                           void* lt_ws, hipStream_t s) {
  int dev = 0;
  hipblasLtHandle_t h = nullptr;
  const fairy2i_status hs = lt_handle(&dev, &h);
  if (hs != FAIRY2I_OK) return hs;
  LtDescs d;
  const int32_t opT = HIPBLAS_OP_T, opN = HIPBLAS_OP_N;
  const int32_t batch = 3;
  const int64_t sa = N * Kp, sb = M * Kp, sc = M * N;
  if (!lt_ok(hipblasLtMatmulDescCreate(&d.op, HIPBLAS_COMPUTE_32F, HIP_R_32F)) ||
      !lt_ok(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_TRANSA, &opT, sizeof(opT))) ||
      !lt_ok(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_TRANSB, &opN, sizeof(opN))) ||
      !lt_ok(hipblasLtMatrixLayoutCreate(&d.a, HIP_R_16BF, (uint64_t)Kp, (uint64_t)N, Kp)) ||
      !lt_ok(hipblasLtMatrixLayoutCreate(&d.b, HIP_R_16BF, (uint64_t)Kp, (uint64_t)M, Kp)) ||
      !lt_ok(hipblasLtMatrixLayoutCreate(&d.c, HIP_R_32F, (uint64_t)N, (uint64_t)M, N)))
    return FAIRY2I_ERR_HIP;
  const hipblasLtMatrixLayout_t lays[3] = {d.a, d.b, d.c};
  const int64_t strides[3] = {sa, sb, sc};
  for (int i = 0; i < 3; ++i)
    if (!lt_ok(hipblasLtMatrixLayoutSetAttribute(lays[i], HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &batch,
                                                 sizeof(batch))) ||
        !lt_ok(hipblasLtMatrixLayoutSetAttribute(lays[i], HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET,
                                                 &strides[i], sizeof(strides[i]))))
      return FAIRY2I_ERR_HIP;
  hipblasLtMatmulAlgo_t algo;
  {
    std::lock_guard<std::mutex> lock(g_lt_mutex);
    const auto key = std::make_tuple(dev, M, N, Kp);
    auto it = g_lt_algos.find(key);
    if (it != g_lt_algos.end()) {
      algo = it->second;
    } else {
      if (!lt_pick(h, d, &algo)) return FAIRY2I_ERR_UNSUPPORTED;
      g_lt_algos[key] = algo;
    }
  }
  const float one = 1.0f, zero = 0.0f;
  if (!lt_ok(hipblasLtMatmul(h, d.op, &one, Bp, d.a, Ap, d.b, &zero, P, d.c, P, d.c, &algo, lt_ws,
                             kLtWorkspaceBytes, s)))
    return FAIRY2I_ERR_HIP;
  return FAIRY2I_OK;
}

// C (row-major M x N, ld ldc, float32) = op(A) op(B), A and B bf16
// row-major: op(A) = A (M x K, ld lda) or A^T (A stored K x M), op(B) = B
// (K x N, ld ldb) or B^T (B stored N x K).  Column-major view for the
// library: C^T (N x M, ld ldc) = op(B)^T op(A)^T, where the stored B is, read
// column-major, op(B)^T itself (no transpose) or its transpose, and A alike.
std::map<std::tuple<int, int64_t, int64_t, int64_t, int, int, int64_t, int64_t, int64_t>, hipblasLtMatmulAlgo_t>
    g_lt_gemm_algos;

// The descriptors of one such problem.
bool lt_gemm_descs(LtDescs& d, int64_t lda, int transA, int64_t ldb, int transB, int64_t M, int64_t N, int64_t K,
                   int64_t ldc) {
  const int32_t opa = transB ? HIPBLAS_OP_T : HIPBLAS_OP_N;  // the library's A is our B
  const int32_t opb = transA ? HIPBLAS_OP_T : HIPBLAS_OP_N;  // and its B our A
  // stored shapes, column-major: B is N x K (no transpose) or K x N; A is K x M or M x K
  const uint64_t ar = transB ? (uint64_t)K : (uint64_t)N, ac = transB ? (uint64_t)N : (uint64_t)K;
  const uint64_t br = transA ? (uint64_t)M : (uint64_t)K, bc = transA ? (uint64_t)K : (uint64_t)M;
  if (!lt_ok(hipblasLtMatmulDescCreate(&d.op, HIPBLAS_COMPUTE_32F, HIP_R_32F)) ||
      !lt_ok(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_TRANSA, &opa, sizeof(opa))) ||
      !lt_ok(hipblasLtMatmulDescSetAttribute(d.op, HIPBLASLT_MATMUL_DESC_TRANSB, &opb, sizeof(opb))) ||
      !lt_ok(hipblasLtMatrixLayoutCreate(&d.a, HIP_R_16BF, ar, ac, ldb)) ||
      !lt_ok(hipblasLtMatrixLayoutCreate(&d.b, HIP_R_16BF, br, bc, lda)) ||
      !lt_ok(hipblasLtMatrixLayoutCreate(&d.c, HIP_R_32F, (uint64_t)N, (uint64_t)M, ldc)))
    return false;
  return true;
}

fairy2i_status lt_gemm(const uint16_t* A, int64_t lda, int transA, const uint16_t* B, int64_t ldb, int transB,
                       int64_t M, int64_t N, int64_t K, float* C, int64_t ldc, void* lt_ws, hipStream_t s) {
  int dev = 0;
  hipblasLtHandle_t h = nullptr;
  const fairy2i_status hs = lt_handle(&dev, &h);
  if (hs != FAIRY2I_OK) return hs;
  LtDescs d;
  if (!lt_gemm_descs(d, lda, transA, ldb, transB, M, N, K, ldc)) return FAIRY2I_ERR_HIP;
  hipblasLtMatmulAlgo_t algo;
  {
    std::lock_guard<std::mutex> lock(g_lt_mutex);
    const auto key = std::make_tuple(dev, M, N, K, transA, transB, lda, ldb, ldc);
    auto it = g_lt_gemm_algos.find(key);
    if (it != g_lt_gemm_algos.end()) {
      algo = it->second;
    } else {
      if (!lt_pick(h, d, &algo)) return FAIRY2I_ERR_UNSUPPORTED;
      g_lt_gemm_algos[key] = algo;
    }
  }
  const float one = 1.0f, zero = 0.0f;
  if (!lt_ok(hipblasLtMatmul(h, d.op, &one, B, d.a, A, d.b, &zero, C, d.c, C, d.c, &algo, lt_ws,
                             kLtWorkspaceBytes, s)))
    return FAIRY2I_ERR_HIP;
  return FAIRY2I_OK;
}

// Up to kTuneCandidates of the library's algorithms for the problem, each
// run twice and then timed over kTuneRuns runs on the stream; the fastest
// is kept for later calls with the same problem.
constexpr int kTuneCandidates = 16;
constexpr int kTuneRuns = 5;

fairy2i_status lt_gemm_tune(const uint16_t* A, int64_t lda, int transA, const uint16_t* B, int64_t ldb, int transB,
                            int64_t M, int64_t N, int64_t K, float* C, int64_t ldc, void* lt_ws, hipStream_t s,
                            float* best_us) {
  int dev = 0;
  hipblasLtHandle_t h = nullptr;
  const fairy2i_status hs = lt_handle(&dev, &h);
  if (hs != FAIRY2I_OK) return hs;
  LtDescs d;
  if (!lt_gemm_descs(d, lda, transA, ldb, transB, M, N, K, ldc)) return FAIRY2I_ERR_HIP;
  hipblasLtMatmulPreference_t pref = nullptr;
  const uint64_t wsb = kLtWorkspaceBytes;
  hipblasLtMatmulHeuristicResult_t res[kTuneCandidates];
  int found = 0;
  const bool ok =
      lt_ok(hipblasLtMatmulPreferenceCreate(&pref)) &&
      lt_ok(hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsb, sizeof(wsb))) &&
      lt_ok(hipblasLtMatmulAlgoGetHeuristic(h, d.op, d.a, d.b, d.c, d.c, pref, kTuneCandidates, res, &found));
  if (pref) hipblasLtMatmulPreferenceDestroy(pref);
  if (!ok || found < 1) return FAIRY2I_ERR_UNSUPPORTED;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    if (e0) (void)hipEventDestroy(e0);
    return FAIRY2I_ERR_HIP;
  }
  const float one = 1.0f, zero = 0.0f;
  int best = -1;
  float best_ms = 0.0f;
  for (int i = 0; i < found; ++i) {
    if (res[i].workspaceSize > kLtWorkspaceBytes) continue;
    bool run_ok = true;
    for (int r = 0; r < 2 && run_ok; ++r)
      run_ok = lt_ok(hipblasLtMatmul(h, d.op, &one, B, d.a, A, d.b, &zero, C, d.c, C, d.c, &res[i].algo, lt_ws,
                                     kLtWorkspaceBytes, s));
    if (!run_ok || hipEventRecord(e0, s) != hipSuccess) continue;
    for (int r = 0; r < kTuneRuns && run_ok; ++r)
      run_ok = lt_ok(hipblasLtMatmul(h, d.op, &one, B, d.a, A, d.b, &zero, C, d.c, C, d.c, &res[i].algo, lt_ws,
                                     kLtWorkspaceBytes, s));
    float ms = 0.0f;
    if (!run_ok || hipEventRecord(e1, s) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
        hipEventElapsedTime(&ms, e0, e1) != hipSuccess)
      continue;
    if (best < 0 || ms < best_ms) {
      best = i;
      best_ms = ms;
    }
  }
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (best < 0) return FAIRY2I_ERR_UNSUPPORTED;
  {
    std::lock_guard<std::mutex> lock(g_lt_mutex);
    g_lt_gemm_algos[std::make_tuple(dev, M, N, K, transA, transB, lda, ldb, ldc)] = res[best].algo;
  }
  if (best_us) *best_us = best_ms * 1e3f / kTuneRuns;
  return FAIRY2I_OK;
}

bool planar_op_ok(const fairy2i_cgemm_operand& o, int64_t rows, int64_t K) {
  if (!o.data) return false;
  if (o.dtype != FAIRY2I_ACT_F32 && o.dtype != FAIRY2I_ACT_BF16) return false;
  if ((o.trans != 0 && o.trans != 1) || (o.conj != 0 && o.conj != 1) || o.reserved != 0) return false;
  return o.trans ? o.ld >= rows : o.ld >= K;
}

// Plane geometry of a call: padded K and the workspace pieces.
struct PlanarGeom {
  int64_t Kp;
  size_t a_bytes, b_bytes, p_bytes, total;
};

bool planar_geom(const int64_t* K, int32_t nseg, int64_t M, int64_t N, PlanarGeom& g) {
  if (!K || nseg < 1 || nseg > 2 || M <= 0 || N <= 0) return false;
  int64_t kt = 0;
  for (int s = 0; s < nseg; ++s) {
    if (K[s] <= 0) return false;
    kt += K[s];
  }
  g.Kp = (kt + kPlaneKAlign - 1) / kPlaneKAlign * kPlaneKAlign;
  g.a_bytes = align256((size_t)3 * M * g.Kp * sizeof(uint16_t));
  g.b_bytes = align256((size_t)3 * N * g.Kp * sizeof(uint16_t));
  g.p_bytes = align256((size_t)3 * M * N * sizeof(float));
  g.total = g.a_bytes + g.b_bytes + g.p_bytes + kLtWorkspaceBytes;
  return true;
}

hipError_t launch_planes(const fairy2i_cgemm_operand* ops, const int64_t* K, int nseg, int64_t rows, int64_t Kp,
                         uint16_t* planes, hipStream_t s) {
  int64_t koff = 0;
  for (int sg = 0; sg < nseg; ++sg) {
    const PlaneOp op{ops[sg].data, ops[sg].ld, ops[sg].dtype, ops[sg].trans, ops[sg].conj, 0};
    // the last segment also writes the zero padding up to Kp
    const int64_t width = sg == nseg - 1 ? Kp - koff : K[sg];
    const dim3 grid((unsigned)((width + kPlaneTile - 1) / kPlaneTile), (unsigned)((rows + kPlaneTile - 1) / kPlaneTile));
    hipLaunchKernelGGL(gauss_planes_kernel, grid, dim3(256), 0, s, op, rows, K[sg], koff, width, Kp, planes);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    koff += K[sg];
  }
  return hipSuccess;
}

}  // namespace

}  // namespace fairy2i

using namespace fairy2i;

extern "C" {

size_t fairy2i_cgemm_gauss_planar_workspace_bytes(const int64_t* K, int32_t nseg, int64_t M, int64_t N) {
  PlanarGeom g;
  if (!planar_geom(K, nseg, M, N, g)) return 0;
  return g.total;
}

fairy2i_status fairy2i_cgemm_gauss_planar(const fairy2i_cgemm_operand* A, const fairy2i_cgemm_operand* B,
                                          const int64_t* K, int32_t nseg, int64_t M, int64_t N, float* C,
                                          int64_t ldc, int32_t accumulate, void* workspace, size_t workspace_bytes,
                                          void* stream) {
  if (!A || !B || !K || !C) return FAIRY2I_ERR_NULL;
  PlanarGeom g;
  if (!planar_geom(K, nseg, M, N, g) || ldc < N || (accumulate != 0 && accumulate != 1)) return FAIRY2I_ERR_SHAPE;
  if (M > 65535LL * kPlaneTile || N > 65535LL * kPlaneTile) return FAIRY2I_ERR_UNSUPPORTED;
  for (int s = 0; s < nseg; ++s) {
    if (!A[s].data || !B[s].data) return FAIRY2I_ERR_NULL;
    if (!planar_op_ok(A[s], M, K[s]) || !planar_op_ok(B[s], N, K[s])) return FAIRY2I_ERR_SHAPE;
  }
  if (!workspace || workspace_bytes < g.total) return FAIRY2I_ERR_WORKSPACE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  auto* Ap = reinterpret_cast<uint16_t*>(ws);
  auto* Bp = reinterpret_cast<uint16_t*>(ws + g.a_bytes);
  auto* P = reinterpret_cast<float*>(ws + g.a_bytes + g.b_bytes);
  void* lt_ws = ws + g.a_bytes + g.b_bytes + g.p_bytes;
  if (launch_planes(A, K, nseg, M, g.Kp, Ap, s) != hipSuccess) return FAIRY2I_ERR_HIP;
  if (launch_planes(B, K, nseg, N, g.Kp, Bp, s) != hipSuccess) return FAIRY2I_ERR_HIP;
  const fairy2i_status st = lt_products(Ap, Bp, P, M, N, g.Kp, lt_ws, s);
  if (st != FAIRY2I_OK) return st;
  const int64_t bx = (N + 255) / 256 < 64 ? (N + 255) / 256 : 64;
  const int64_t by = M < 16384 ? M : 16384;
  hipLaunchKernelGGL(gauss_combine_kernel, dim3((unsigned)bx, (unsigned)by), dim3(256), 0, s, P, M, N,
                     reinterpret_cast<float2*>(C), ldc, accumulate);
  return hipGetLastError() == hipSuccess ? FAIRY2I_OK : FAIRY2I_ERR_HIP;
}

size_t fairy2i_gemm_bf16_workspace_bytes(void) { return kLtWorkspaceBytes; }

fairy2i_status fairy2i_gemm_bf16_tune(const void* A, int64_t lda, int32_t transA, const void* B, int64_t ldb,
                                      int32_t transB, int64_t M, int64_t N, int64_t K, float* C, int64_t ldc,
                                      void* workspace, size_t workspace_bytes, float* best_us, void* stream) {
  if (!A || !B || !C) return FAIRY2I_ERR_NULL;
  if ((transA != 0 && transA != 1) || (transB != 0 && transB != 1)) return FAIRY2I_ERR_SHAPE;
  if (M <= 0 || N <= 0 || K <= 0 || ldc < N) return FAIRY2I_ERR_SHAPE;
  if (lda < (transA ? M : K) || ldb < (transB ? K : N)) return FAIRY2I_ERR_SHAPE;
  if (!workspace || workspace_bytes < kLtWorkspaceBytes) return FAIRY2I_ERR_WORKSPACE;
  return lt_gemm_tune(static_cast<const uint16_t*>(A), lda, transA, static_cast<const uint16_t*>(B), ldb, transB, M,
                      N, K, C, ldc, workspace, static_cast<hipStream_t>(stream), best_us);
}

fairy2i_status fairy2i_gemm_bf16(const void* A, int64_t lda, int32_t transA, const void* B, int64_t ldb,
                                 int32_t transB, int64_t M, int64_t N, int64_t K, float* C, int64_t ldc,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  if (!A || !B || !C) return FAIRY2I_ERR_NULL;
  if ((transA != 0 && transA != 1) || (transB != 0 && transB != 1)) return FAIRY2I_ERR_SHAPE;
  if (M <= 0 || N <= 0 || K <= 0 || ldc < N) return FAIRY2I_ERR_SHAPE;
  if (lda < (transA ? M : K) || ldb < (transB ? K : N)) return FAIRY2I_ERR_SHAPE;
  if (!workspace || workspace_bytes < kLtWorkspaceBytes) return FAIRY2I_ERR_WORKSPACE;
  return lt_gemm(static_cast<const uint16_t*>(A), lda, transA, static_cast<const uint16_t*>(B), ldb, transB, M, N,
                 K, C, ldc, workspace, static_cast<hipStream_t>(stream));
}

}  // extern "C"
