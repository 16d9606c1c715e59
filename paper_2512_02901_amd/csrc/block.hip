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
// Complex vectors are float2 (re, im); a head owns dc = n / n_heads
// consecutive complex entries (entry j: its real dims j and j + dc).  All
// reductions run in a fixed order, so results are bitwise reproducible.
#include <math.h>
#include <string.h>

#include "common.h"

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

// One wave per (64-position slice, head).  Lane t scores position n0 + t as
// Re(q^H k) * scale, reading its key with 16-byte loads and the query from
// LDS (every lane reads the same address: a broadcast); then the slice's
// maximum m, e_t = exp(s_t - m), l = sum e_t; then lane j forms
// o_j = sum_t e_t v_{n0+t, j} over the slice (t wave-uniform, eight value loads
// in flight).  Partial record per (head, slice): [m, l, o (2 dc floats)].
template <int R>  // complex entries per lane in the value pass: dc <= 64 R
__global__ __launch_bounds__(64) void attn_partial_kernel(const float2* __restrict__ q_rot,
                                                          const float2* __restrict__ k_cache,
                                                          const float2* __restrict__ v_cache, int dc, int64_t n_ctx,
                                                          int64_t max_ctx, float scale, float* __restrict__ part) {
  __shared__ float4 qs[64 * R / 2];
  const int h = blockIdx.y, sl = blockIdx.x, lane = threadIdx.x;
  const int64_t n0 = (int64_t)sl * kAttnSlice;
  const int cnt = (int)min((int64_t)kAttnSlice, n_ctx - n0);
  for (int j = lane; j < dc / 2; j += 64) qs[j] = reinterpret_cast<const float4*>(q_rot + h * dc)[j];
  __syncthreads();
  const float2* kh = k_cache + (int64_t)h * max_ctx * dc;
  const float2* vh = v_cache + (int64_t)h * max_ctx * dc;
  float s = -INFINITY;
  if (lane < cnt) {
    const float4* kp = reinterpret_cast<const float4*>(kh + (n0 + lane) * dc);
    float acc = 0.0f;
    for (int j0 = 0; j0 < dc / 2; j0 += 8) {
      float4 kv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) kv[u] = j0 + u < dc / 2 ? kp[j0 + u] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        if (j0 + u < dc / 2) {
          const float4 qv = qs[j0 + u];
          acc = fmaf(qv.x, kv[u].x, acc);
          acc = fmaf(qv.y, kv[u].y, acc);
          acc = fmaf(qv.z, kv[u].z, acc);
          acc = fmaf(qv.w, kv[u].w, acc);
        }
      }
    }
    s = acc * scale;
  }
  const float m = wave_max(s);
  const float e = lane < cnt ? expf(s - m) : 0.0f;
  const float l = wave_sum(e);
  float2 o[R];
#pragma unroll
  for (int r = 0; r < R; ++r) o[r] = make_float2(0.f, 0.f);
  for (int t0 = 0; t0 < cnt; t0 += 8) {
    float2 vv[8][R];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int j = lane + 64 * r;
        vv[u][r] = (t0 + u < cnt && j < dc) ? vh[(n0 + t0 + u) * dc + j] : make_float2(0.f, 0.f);
      }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      // lanes t >= cnt hold e = 0, and t0 + u < 64
      const float w = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(e), t0 + u));
#pragma unroll
      for (int r = 0; r < R; ++r) {
        o[r].x = fmaf(w, vv[u][r].x, o[r].x);
        o[r].y = fmaf(w, vv[u][r].y, o[r].y);
      }
    }
  }
  float* rec = part + ((int64_t)h * gridDim.x + sl) * (2 + 2 * dc);
  if (lane == 0) {
    rec[0] = m;
    rec[1] = l;
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = lane + 64 * r;
    if (j < dc) {
      rec[2 + 2 * j] = o[r].x;
      rec[3 + 2 * j] = o[r].y;
    }
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

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Plan: header, then the four group tables (q k v; o; gate up; down).
constexpr uint32_t kBlockMagic = 0xFA11B10Cu;
constexpr int kGroups = 4;
struct BlockPlanHeader {
  uint32_t magic, abi;
  int64_t n, n_ff, max_ctx;
  int32_t n_heads, T;
  float eps;
  int32_t pad0_;
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
  hipLaunchKernelGGL(add_rmsnorm_kernel, dim3(1), dim3(kNormThreads), 0, s, xin, nullptr, nullptr, hdr->norm_attn,
                     hdr->eps, n, hdr->z);
  if ((e = hipGetLastError()) != hipSuccess) return hip_st(e);
  if ((st = group(0)) != FAIRY2I_OK) return st;
  hipLaunchKernelGGL(rope_append_kernel, dim3((n + 255) / 256), dim3(256), 0, s, hdr->q, hdr->k, hdr->v, n, dc, pos,
                     hdr->max_ctx, hdr->rope_base, hdr->q_rot, kc, vc);
  const float scale = (float)(1.0 / sqrt((double)(2 * dc)));
  if (dc <= 64)
    hipLaunchKernelGGL(attn_partial_kernel<1>, dim3(slices, H), dim3(64), 0, s, hdr->q_rot, kc, vc, dc, n_ctx,
                       hdr->max_ctx, scale, hdr->part);
  else
    hipLaunchKernelGGL(attn_partial_kernel<4>, dim3(slices, H), dim3(64), 0, s, hdr->q_rot, kc, vc, dc, n_ctx,
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
