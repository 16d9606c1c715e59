// Decode product (1..16 tokens) on the int8 matrix cores, for bf16 and int8
// activations.  Sec. 3.4 / Algorithm 1 with the dequantisation of
// Eq. (ifairy-dequant) and the W conj(x) term of Eq. (widely-linear).
//
// Per code i^k the real 2x2 block is b_re I + b_im J (Eq. realify-ops) with
// ternary (b_re, b_im); the two axis planes are contracted separately because
// their scales differ.  Each 32-bit word of 16 codes is expanded in
// registers into the int8 b_re and b_im planes with two v_perm byte-table
// lookups per 4 codes (about one VALU instruction per code), and
// v_mfma_i32_16x16x64_i8 multiplies them with the activations:
//     D[x column][weight row] = sum_j X[j][x column] * B_p[row][j].
// The activation operand carries, per token, the columns
//   int8 activations:  (q_re, q_im)                         -> 8 tokens per 16 columns
//   bf16 activations:  the 3 base-256 digits of X_re, X_im  -> 2 tokens per 16 columns
// where X = rint(x * 2^E) is the token's 23-bit block fixed-point form
// (E chosen per token so that max |X| < 2^22; every bf16 value within 2^14 of
// the token's largest magnitude is represented exactly, smaller ones are
// rounded to the 2^-E grid).  The integer products are exact; digits are
// recombined in int64 and the axis scales, the factor i, the conjugation of
// the W term and the token scale 2^-E (or the int8 dequantisation factor) are
// applied once per output in double, then rounded to float32.
//
// Work item = (layer, 16 weight rows, 512-code slice of K).  A wave loads the
// 2T code planes of its item with one 16-byte load per lane and plane per
// 256 codes, all issued before any arithmetic.  Items of the same rows are
// adjacent, so concurrently running waves read contiguous 8 KB runs of each
// plane.  When K spans several slices, each item writes a float32 partial
// and a second kernel sums the partials in slice order, so results do not
// depend on scheduling.  A table of layers is processed by one launch of
// each kernel (used for a whole decoder stack).
#include "common.h"
#include "decode.h"

namespace fairy2i {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr uint32_t kTableRe = 0x00FF0001u;  // code 0 -> +1, 1 -> 0, 2 -> -1, 3 -> 0
constexpr uint32_t kTableIm = 0xFF000100u;  // code 0 -> 0, 1 -> +1, 2 -> 0, 3 -> -1

__device__ inline void expand_codes(uint32_t w, v4i& bre, v4i& bim) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const uint32_t sel = (w >> (2 * c)) & 0x03030303u;
    bre[c] = (int)__builtin_amdgcn_perm(0u, kTableRe, sel);
    bim[c] = (int)__builtin_amdgcn_perm(0u, kTableIm, sel);
  }
}

__device__ inline int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ inline int64_t uniform64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Layer of an item (wave-uniform): the last layer whose first item is <= item.
__device__ inline int find_layer(const DecLayer* tab, int n, int64_t item) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (uniform64(tab[mid].item0) <= item) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// A descriptor from the table, with every field forced wave-uniform so that
// pointers and buffer descriptors live in scalar registers.
__device__ inline DecLayer load_layer(const DecLayer* p) {
  DecLayer out;
  const uint32_t* src = reinterpret_cast<const uint32_t*>(p);
  uint32_t* dst = reinterpret_cast<uint32_t*>(&out);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(DecLayer) / 4); ++i) dst[i] = __builtin_amdgcn_readfirstlane(src[i]);
  return out;
}

// Column of a 16-column activation tile -> (token, digit/component) or invalid.
template <int MODE>
__device__ inline bool col_token(int tile, int col, int B, int& b, int& digit, int& comp) {
  if constexpr (MODE == kModeBf16) {
    b = 2 * tile + (col >> 3);
    const int ci = col & 7;
    digit = ci >> 1;
    comp = ci & 1;
    return ci < 6 && b < B;
  } else {
    b = 8 * tile + (col >> 1);
    digit = 0;
    comp = col & 1;
    return b < B;
  }
}

// ----------------------------------------------------------------- prep ---
// One block per (tile, column) and layer: writes that column of the
// activation operand for every 64-code MFMA step, in the lane order the
// decode kernel loads (16 bytes per lane, byte 4c+b = code c + 4b of the
// lane's 16-code group), and the per-token scale.
template <int MODE>
__global__ __launch_bounds__(256) void dec_prep_kernel(DecHeader h, DecLayer inl,
                                                       const DecLayer* __restrict__ tab) {
  const DecLayer L = tab ? load_layer(tab + blockIdx.y) : inl;
  const int tile = blockIdx.x >> 4, col = blockIdx.x & 15;
  int b, digit, comp;
  if (!col_token<MODE>(tile, col, h.B, b, digit, comp)) return;
  const int64_t K = L.K;
  __shared__ float red[4];
  __shared__ int sh_E;
  int E = 0;
  if constexpr (MODE == kModeBf16) {
    const uint16_t* xb = static_cast<const uint16_t*>(L.x) + (int64_t)b * K * 2;
    float m = 0.0f;
    for (int64_t i = threadIdx.x; i < 2 * K; i += blockDim.x)
      m = fmaxf(m, fabsf(__uint_as_float((uint32_t)xb[i] << 16)));
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
      const float g = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
      int ex = 0;
      if (g > 0.0f) {
        frexpf(g, &ex);       // g in [2^(ex-1), 2^ex)
        E = 22 - ex;          // g * 2^E in [2^21, 2^22)
        if (E > 149) E = 149; // keep 2^-E representable in float32
      }
      sh_E = E;
      if (digit == 0 && comp == 0) L.xs[b] = g > 0.0f ? ldexpf(1.0f, -E) : 0.0f;
    }
    __syncthreads();
    E = sh_E;
  } else {
    // the accumulator export passes no factors (its epilogue does not use them)
    if (threadIdx.x == 0 && comp == 0) L.xs[b] = L.x_scale_in ? L.x_scale_in[b] : 1.0f;
  }
  const int nchunks = L.nk4 * 16;  // (k4, d, g)
  for (int ch = threadIdx.x; ch < nchunks; ch += blockDim.x) {
    const int kk = ch >> 4, d = (ch >> 2) & 3, g = ch & 3;
    const int64_t k0 = (int64_t)kk * 256 + 64 * g + 16 * d;
    uint32_t out[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int dd = e >> 2, bb = e & 3;
      const int64_t k = k0 + dd + 4 * bb;
      int v = 0;
      if (k < K) {
        if constexpr (MODE == kModeBf16) {
          const uint16_t raw = static_cast<const uint16_t*>(L.x)[((int64_t)b * K + k) * 2 + comp];
          const int X = (int)rintf(ldexpf(__uint_as_float((uint32_t)raw << 16), E));
          const int d0 = ((X + 128) & 255) - 128;
          const int X1 = (X - d0) >> 8;
          const int d1 = ((X1 + 128) & 255) - 128;
          const int d2 = (X1 - d1) >> 8;
          v = digit == 0 ? d0 : (digit == 1 ? d1 : d2);
        } else {
          v = static_cast<const int8_t*>(L.x)[((int64_t)b * K + k) * 2 + comp];
        }
      }
      out[dd] |= ((uint32_t)v & 0xFFu) << (8 * bb);
    }
    const int lane = g * 16 + col;
    uint4* dst = reinterpret_cast<uint4*>(L.xf + ((((int64_t)tile * L.nk4 + kk) * 4 + d) * 64 + lane) * 16);
    *dst = make_uint4(out[0], out[1], out[2], out[3]);
  }
}

// --------------------------------------------------------------- decode ---
constexpr uint32_t kOob = 0xFFFFFFF0u;  // buffer offset past every range: loads return 0

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ inline v4i buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

template <int MODE, int T, int NTG, bool EXPORT>
__global__ __launch_bounds__(256) void dec_mfma_kernel(DecHeader h, DecLayer inl,
                                                       const DecLayer* __restrict__ tab) {
  constexpr int P = 2 * T;  // code planes (M, t)
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int g = lane >> 4, li = lane & 15;
  const int64_t nwaves = (int64_t)gridDim.x * 4;

  for (int64_t item = (int64_t)blockIdx.x * 4 + wave; item < h.total_items; item += nwaves) {
    item = uniform64(item);
    const DecLayer L = tab ? load_layer(tab + find_layer(tab, h.n_layers, item)) : inl;
    const int64_t local = item - L.item0;
    const int rb = (int)(local / L.nkc), kc = (int)(local % L.nkc);
    const int N = L.N, K = L.K;
    const uint32_t plane_bytes = (uint32_t)((int64_t)N * K / 4);
    const int row = rb * 16 + li;
    const bool row_ok = row < N;
    const int k4b = kc * kDecKc4;
    const int nk4_item = min(kDecKc4, L.nk4 - k4b);  // wave-uniform

    const uint32_t xf_bytes = (uint32_t)(h.ntile * L.nk4 * 4 * 64 * 16);
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(L.xf, xf_bytes);

    // Usually one pass (all tiles fit one group); further passes re-read the
    // item's codes, which are then cache hits.
    for (int tg0 = 0; tg0 < h.ntile; tg0 += NTG) {
      // ---- every load of the pass first (out-of-range lanes read 0) ----
      v4i cw[P][kDecKc4];
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const int m = p / T, t = p % T;
        const __amdgpu_buffer_rsrc_t rs = make_rsrc(L.codes[m] + (int64_t)t * plane_bytes, plane_bytes);
#pragma unroll
        for (int j = 0; j < kDecKc4; ++j) {
          const int kk = k4b + j;
          const bool ok = row_ok && j < nk4_item && kk * 256 + 64 * g < K;
          const uint32_t off = ok ? (uint32_t)row * (uint32_t)(K / 4) + (uint32_t)(kk * 64 + 16 * g) : kOob;
          cw[p][j] = buf_load16(rs, off);
        }
      }
      v4i xa[kDecKc4][4][NTG];
#pragma unroll
      for (int j = 0; j < kDecKc4; ++j)
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int tt = 0; tt < NTG; ++tt) {
            const int tile = tg0 + tt, kk = k4b + j;
            int b, digit, comp;
            const bool ok = j < nk4_item && tile < h.ntile && col_token<MODE>(tile, li, h.B, b, digit, comp);
            const uint32_t off = ok ? (uint32_t)((((tile * L.nk4 + kk) * 4 + d) * 64 + lane) * 16) : kOob;
            xa[j][d][tt] = buf_load16(xr, off);
          }

      v4i acc[P][2][NTG];
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int ax = 0; ax < 2; ++ax)
#pragma unroll
          for (int tt = 0; tt < NTG; ++tt) acc[p][ax][tt] = v4i{0, 0, 0, 0};

#pragma unroll
      for (int j = 0; j < kDecKc4; ++j) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
#pragma unroll
          for (int p = 0; p < P; ++p) {
            v4i bre, bim;
            expand_codes((uint32_t)cw[p][j][d], bre, bim);
#pragma unroll
            for (int tt = 0; tt < NTG; ++tt) {
              acc[p][0][tt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(xa[j][d][tt], bre, acc[p][0][tt], 0, 0, 0);
              acc[p][1][tt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(xa[j][d][tt], bim, acc[p][1][tt], 0, 0, 0);
            }
            // keep each plane's expansion next to its MFMAs (bounds live registers)
            __builtin_amdgcn_sched_group_barrier(0x002, 15, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 2 * NTG, 0);
          }
        }
      }

      // ---- epilogue: lane holds x columns 4g..4g+3 of weight row li ----
#pragma unroll
      for (int tt = 0; tt < NTG; ++tt) {
        const int tile = tg0 + tt;
        // bf16: token 2*tile + g/2 has digits 0, 1 in group g and digit 2 in
        // group g+1; fetch the latter (all lanes take part in the shuffle).
        int hi[P][2][2];
        if constexpr (MODE == kModeBf16) {
#pragma unroll
          for (int p = 0; p < P; ++p)
#pragma unroll
            for (int ax = 0; ax < 2; ++ax) {
              hi[p][ax][0] = __shfl_down(acc[p][ax][tt][0], 16);
              hi[p][ax][1] = __shfl_down(acc[p][ax][tt][1], 16);
            }
        }
        if (!row_ok || tile >= h.ntile) continue;
        const int ntok = MODE == kModeBf16 ? ((g & 1) ? 0 : 1) : 2;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          if (s >= ntok) break;
          const int b = MODE == kModeBf16 ? 2 * tile + (g >> 1) : 8 * tile + 2 * g + s;
          if (b >= h.B) continue;
          // exact integer product of plane (p, ax) with component c of token b
          auto Pv = [&](int p, int ax, int c) -> int64_t {
            if constexpr (MODE == kModeBf16)
              return (int64_t)acc[p][ax][tt][c] + 256 * (int64_t)acc[p][ax][tt][2 + c] +
                     65536 * (int64_t)hi[p][ax][c];
            else
              return (int64_t)acc[p][ax][tt][2 * s + c];
          };
          if constexpr (EXPORT) {
#pragma unroll
            for (int p = 0; p < P; ++p)
#pragma unroll
              for (int ax = 0; ax < 2; ++ax) {
                int32_t* dst = L.acc + ((((int64_t)p * 2 + ax) * h.B + b) * N + row) * 2;
                atomicAdd(dst, (int32_t)Pv(p, ax, 0));
                atomicAdd(dst + 1, (int32_t)Pv(p, ax, 1));
              }
          } else {
            double yr = 0.0, yi = 0.0;
#pragma unroll
            for (int t = 0; t < T; ++t) {
              const double su_re = L.scales[0][2 * t], su_im = L.scales[0][2 * t + 1];
              const double sw_re = L.scales[1][2 * t], sw_im = L.scales[1][2 * t + 1];
              const int pu = t, pw = T + t;
              yr += su_re * (double)Pv(pu, 0, 0) - su_im * (double)Pv(pu, 1, 1);
              yi += su_re * (double)Pv(pu, 0, 1) + su_im * (double)Pv(pu, 1, 0);
              yr += sw_re * (double)Pv(pw, 0, 0) + sw_im * (double)Pv(pw, 1, 1);
              yi += -sw_re * (double)Pv(pw, 0, 1) + sw_im * (double)Pv(pw, 1, 0);
            }
            const double f = (double)L.xs[b];
            const float2 v = make_float2((float)(yr * f), (float)(yi * f));
            if (L.nkc == 1)
              L.y[(int64_t)b * N + row] = v;
            else
              L.part[((int64_t)kc * h.B + b) * N + row] = v;
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------ reduction ---
__global__ __launch_bounds__(256) void dec_reduce_kernel(DecHeader h, DecLayer inl,
                                                         const DecLayer* __restrict__ tab) {
  const DecLayer L = tab ? load_layer(tab + blockIdx.y) : inl;
  if (L.nkc <= 1) return;
  const int64_t n = (int64_t)h.B * L.N;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    float re = 0.0f, im = 0.0f;
    for (int kc = 0; kc < L.nkc; ++kc) {
      const float2 v = L.part[(int64_t)kc * n + i];
      re += v.x;
      im += v.y;
    }
    L.y[i] = make_float2(re, im);
  }
}

__global__ void fill_i32_kernel(int32_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

template <int MODE, int T, int NTG, bool EXPORT>
void launch_dec(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, int blocks,
                hipStream_t s) {
  hipLaunchKernelGGL((dec_mfma_kernel<MODE, T, NTG, EXPORT>), dim3(blocks), dim3(256), 0, s, h, inl, tab);
}

template <int MODE, bool EXPORT>
void launch_dec_mode(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, int blocks,
                     hipStream_t s) {
  const int ntg = dec_tiles_per_group(h.T, h.ntile);
  switch (h.T * 8 + ntg) {
    case 1 * 8 + 1: launch_dec<MODE, 1, 1, EXPORT>(h, inl, tab, blocks, s); break;
    case 1 * 8 + 2: launch_dec<MODE, 1, 2, EXPORT>(h, inl, tab, blocks, s); break;
    case 1 * 8 + 4: launch_dec<MODE, 1, 4, EXPORT>(h, inl, tab, blocks, s); break;
    case 2 * 8 + 1: launch_dec<MODE, 2, 1, EXPORT>(h, inl, tab, blocks, s); break;
    case 2 * 8 + 2: launch_dec<MODE, 2, 2, EXPORT>(h, inl, tab, blocks, s); break;
    case 2 * 8 + 4: launch_dec<MODE, 2, 4, EXPORT>(h, inl, tab, blocks, s); break;
    case 3 * 8 + 1: launch_dec<MODE, 3, 1, EXPORT>(h, inl, tab, blocks, s); break;
    case 3 * 8 + 2: launch_dec<MODE, 3, 2, EXPORT>(h, inl, tab, blocks, s); break;
    case 4 * 8 + 1: launch_dec<MODE, 4, 1, EXPORT>(h, inl, tab, blocks, s); break;
    default: launch_dec<MODE, 4, 2, EXPORT>(h, inl, tab, blocks, s); break;
  }
}

}  // namespace

int dec_tiles_per_group(int T, int ntile) {
  const int cap = T <= 2 ? 4 : 2;
  int ntg = 1;
  while (ntg < ntile && ntg < cap) ntg *= 2;
  return ntg;
}

hipError_t launch_decode(const DecHeader& h, const DecLayer& inl, const DecLayer* tab,
                         int any_split, int64_t max_BN, bool export_acc, int64_t acc_elems,
                         int32_t* acc, hipStream_t s, hipEvent_t const* events) {
  const int nl = h.n_layers;
  auto mark = [&](int i) -> hipError_t { return events ? hipEventRecord(events[i], s) : hipSuccess; };
  hipError_t e = mark(0);
  if (e != hipSuccess) return e;
  // 1. activation operand
  if (h.mode == kModeBf16)
    hipLaunchKernelGGL(dec_prep_kernel<kModeBf16>, dim3(h.ntile * 16, nl), dim3(256), 0, s, h, inl, tab);
  else
    hipLaunchKernelGGL(dec_prep_kernel<kModeI8>, dim3(h.ntile * 16, nl), dim3(256), 0, s, h, inl, tab);
  if ((e = hipGetLastError()) != hipSuccess || (e = mark(1)) != hipSuccess) return e;
  if (export_acc) {
    hipLaunchKernelGGL(fill_i32_kernel, dim3(1024), dim3(256), 0, s, acc, acc_elems);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // 2. products
  int64_t blocks = (h.total_items + 3) / 4;
  if (blocks > kDecMaxBlocks) blocks = kDecMaxBlocks;
  if (h.mode == kModeBf16) {
    launch_dec_mode<kModeBf16, false>(h, inl, tab, (int)blocks, s);
  } else if (export_acc) {
    launch_dec_mode<kModeI8, true>(h, inl, tab, (int)blocks, s);
  } else {
    launch_dec_mode<kModeI8, false>(h, inl, tab, (int)blocks, s);
  }
  if ((e = hipGetLastError()) != hipSuccess || (e = mark(2)) != hipSuccess) return e;
  // 3. split-K partials, summed in slice order
  if (!export_acc && any_split) {
    int64_t rb = (max_BN + 255) / 256;
    if (rb > 4096) rb = 4096;
    hipLaunchKernelGGL(dec_reduce_kernel, dim3((unsigned)rb, nl), dim3(256), 0, s, h, inl, tab);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return mark(3);
}

}  // namespace fairy2i

namespace fairy2i {

namespace {
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
}  // namespace

size_t dec_layer_setup(DecLayer& l, int T, int mode, int B, char* ws) {
  (void)T;
  const int ntile = mode == kModeBf16 ? (B + 1) / 2 : (B + 7) / 8;
  l.nrb = (int32_t)((l.N + 15) / 16);
  l.nk4 = (int32_t)((l.K + 255) / 256);
  l.nkc = (l.nk4 + kDecKc4 - 1) / kDecKc4;
  const size_t xf_bytes = align256((size_t)ntile * l.nk4 * 4 * 64 * 16);
  const size_t xs_bytes = align256((size_t)B * sizeof(float));
  const size_t part_bytes = l.nkc > 1 ? align256((size_t)l.nkc * B * l.N * sizeof(float2)) : 0;
  if (ws) {
    l.xf = reinterpret_cast<int8_t*>(ws);
    l.xs = reinterpret_cast<float*>(ws + xf_bytes);
    l.part = part_bytes ? reinterpret_cast<float2*>(ws + xf_bytes + xs_bytes) : nullptr;
  }
  return xf_bytes + xs_bytes + part_bytes;
}

}  // namespace fairy2i
