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
#include <type_traits>

#include "common.h"
#include "decode.h"

namespace fairy2i {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

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

// Scalar (SMEM) loads of wave-uniform operands.  Scalar loads are tracked by
// lgkmcnt, so waiting for them does not drain the vector-memory queue that
// holds the prefetched code bytes.

typedef float sf2 __attribute__((ext_vector_type(2)));
typedef float sf4 __attribute__((ext_vector_type(4)));
typedef float sf8 __attribute__((ext_vector_type(8)));

// Axis scales of both matrices, sc[m][t][axis], by scalar loads that are all
// in flight before one wait.  The arrays hold exactly 2T floats each.
template <int T>
__device__ inline void sload_scales(const float* pu, const float* pw, float (&sc)[2][T][2]) {
  float a[2][2 * T];
  if constexpr (T == 1) {
    sf2 u, w;
    __asm__ volatile("s_load_dwordx2 %0, %2, 0x0\n\ts_load_dwordx2 %1, %3, 0x0\n\ts_waitcnt lgkmcnt(0)"
                     : "=&s"(u), "=&s"(w) : "s"(pu), "s"(pw) : "memory");
    for (int i = 0; i < 2; ++i) { a[0][i] = u[i]; a[1][i] = w[i]; }
  } else if constexpr (T == 2) {
    sf4 u, w;
    __asm__ volatile("s_load_dwordx4 %0, %2, 0x0\n\ts_load_dwordx4 %1, %3, 0x0\n\ts_waitcnt lgkmcnt(0)"
                     : "=&s"(u), "=&s"(w) : "s"(pu), "s"(pw) : "memory");
    for (int i = 0; i < 4; ++i) { a[0][i] = u[i]; a[1][i] = w[i]; }
  } else if constexpr (T == 3) {
    sf4 u, w;
    sf2 u2, w2;
    __asm__ volatile(
        "s_load_dwordx4 %0, %4, 0x0\n\ts_load_dwordx2 %1, %4, 0x10\n\t"
        "s_load_dwordx4 %2, %5, 0x0\n\ts_load_dwordx2 %3, %5, 0x10\n\ts_waitcnt lgkmcnt(0)"
        : "=&s"(u), "=&s"(u2), "=&s"(w), "=&s"(w2) : "s"(pu), "s"(pw) : "memory");
    for (int i = 0; i < 4; ++i) { a[0][i] = u[i]; a[1][i] = w[i]; }
    for (int i = 0; i < 2; ++i) { a[0][4 + i] = u2[i]; a[1][4 + i] = w2[i]; }
  } else {
    static_assert(T == 4, "1 <= T <= 4");
    sf8 u, w;
    __asm__ volatile("s_load_dwordx8 %0, %2, 0x0\n\ts_load_dwordx8 %1, %3, 0x0\n\ts_waitcnt lgkmcnt(0)"
                     : "=&s"(u), "=&s"(w) : "s"(pu), "s"(pw) : "memory");
    for (int i = 0; i < 8; ++i) { a[0][i] = u[i]; a[1][i] = w[i]; }
  }
#pragma unroll
  for (int m = 0; m < 2; ++m)
#pragma unroll
    for (int t = 0; t < T; ++t) {
      sc[m][t][0] = a[m][2 * t];
      sc[m][t][1] = a[m][2 * t + 1];
    }
}

// NT consecutive floats (2 or 8) at a wave-uniform address, one scalar load.
// The caller guarantees the NT floats lie inside the allocation.
template <int NT>
__device__ inline void sload_run(const float* p, float (&v)[NT]) {
  if constexpr (NT == 2) {
    sf2 r;
    __asm__ volatile("s_load_dwordx2 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=&s"(r) : "s"(p) : "memory");
    v[0] = r[0];
    v[1] = r[1];
  } else {
    static_assert(NT == 8, "2 or 8 floats");
    sf8 r;
    __asm__ volatile("s_load_dwordx8 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=&s"(r) : "s"(p) : "memory");
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = r[i];
  }
}

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
// pointers and buffer descriptors live in scalar registers.  Field by field,
// so the copy never goes through memory.
template <typename P>
__device__ inline P* uniform_ptr(P* v) {
  return reinterpret_cast<P*>(uniform64(reinterpret_cast<int64_t>(v)));
}

__device__ inline DecLayer load_layer(const DecLayer* p) {
  DecLayer o;
  o.codes[0] = uniform_ptr(p->codes[0]);
  o.codes[1] = uniform_ptr(p->codes[1]);
  o.scales[0] = uniform_ptr(p->scales[0]);
  o.scales[1] = uniform_ptr(p->scales[1]);
  o.x = uniform_ptr(p->x);
  o.x_scale_in = uniform_ptr(p->x_scale_in);
  o.y = uniform_ptr(p->y);
  o.acc = uniform_ptr(p->acc);
  o.xf = uniform_ptr(p->xf);
  o.xs = uniform_ptr(p->xs);
  o.part = uniform_ptr(p->part);
  o.N = uniform(p->N);
  o.K = uniform(p->K);
  o.nrb = uniform(p->nrb);
  o.nk4 = uniform(p->nk4);
  o.nkc = uniform(p->nkc);
  o.kc4 = uniform(p->kc4);
  o.tiled = uniform(p->tiled);
  o.pad_ = 0;
  o.item0 = uniform64(p->item0);
  return o;
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
  } else if constexpr (MODE == kModeBf16F4) {
    b = 2 * tile + (col >> 3);  // columns 8b' .. 8b'+7: (digit, component) of token b'
    digit = (col >> 1) & 3;
    comp = col & 1;
    return b < B;
  } else {
    b = 8 * tile + (col >> 1);
    digit = 0;
    comp = col & 1;
    return b < B;
  }
}

// --------------------------------------------------------------- decode ---
constexpr uint32_t kOob = 0xFFFFFFF0u;  // buffer offset past every range: loads return 0
constexpr int kNonTemporal = 2;         // buffer-load cache policy: streaming (nt), for bytes read once

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ inline v4i buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

typedef float v2f __attribute__((ext_vector_type(2)));
__device__ inline void buf_store8(const void* base, uint32_t bytes, uint32_t off, float2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(v2f{v.x, v.y}, make_rsrc(base, bytes), off, 0, 0);
}

// ----------------------------------------------------------------- prep ---
// Layout of the activation operand: [tile][256-code step][d][g][column < nc]
// [16 bytes].  Int8 operand: the 16 bytes of (column, g, d) are what the
// MFMA lane of that column and 16-code group g takes for the step's d-th
// 64-code MFMA (byte 4c+b = code c + 4b of the group).  Fp8 operand (the fp4
// code layout): they are bytes 16 (d % 2) .. +15 of what the lane of that
// column and lane group g takes for the step's (d / 2)-th 128-code MFMA, the
// activations of codes 64 d + 16 g .. +15 of the step.  The nc columns of a
// step are contiguous, so a step's whole operand is one nc * 256-byte run.
// Columns that hold no token are written as zeros.

// 16 consecutive complex activations x[b][k0 .. k0+15] of one component as
// raw bits (bf16: 16-bit patterns, int8: sign-extended bytes).  Vector loads
// when the activation pointer allows them.
constexpr int kPrepSplit = 4;

// The e4m3 (OCP fp8: 1 sign, 4 exponent bits with bias 7, 3 mantissa bits)
// encoding of an integer |d| <= 16, which it represents exactly.
__device__ inline uint32_t e4m3_of_int(int d) {
  const uint32_t a = (uint32_t)(d < 0 ? -d : d);
  if (a == 0) return 0u;
  const int ex = 31 - __builtin_clz(a);  // a = 1.m * 2^ex
  return (d < 0 ? 0x80u : 0u) | ((uint32_t)(ex + 7) << 3) | (((a << 3) >> ex) & 7u);
}

template <int MODE>
__device__ inline void load_run16(const void* x, bool vec, int64_t e0, int comp, int (&v)[16]) {
  if constexpr (MODE == kModeBf16) {
    const uint16_t* p = static_cast<const uint16_t*>(x) + e0;
    if (vec) {
      const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint4 w = q[i];
        const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) v[4 * i + j] = (int)(comp ? wd[j] >> 16 : wd[j] & 0xFFFFu);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] = p[2 * i + comp];
    }
  } else {
    const int8_t* p = static_cast<const int8_t*>(x) + e0;
    if (vec) {
      const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const uint4 w = q[i];
        const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          v[8 * i + 2 * j] = (int)(int8_t)(wd[j] >> (8 * comp));
          v[8 * i + 2 * j + 1] = (int)(int8_t)(wd[j] >> (16 + 8 * comp));
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < 16; ++i) v[i] = p[2 * i + comp];
    }
  }
}

// kPrepSplit blocks per (activation tile, layer).  bf16: each block first
// finds the block fixed-point exponent of the tile's two tokens (from their
// largest magnitudes), then writes its share of the tile's 16-byte operand
// chunks, one chunk per thread in storage order.  int8: the bytes are copied into place and the per-token
// dequantisation factors passed on.
template <int MODE>
__global__ __launch_bounds__(256) void dec_prep_kernel(DecHeader h, DecLayer inl,
                                                       const DecLayer* __restrict__ tab) {
  const DecLayer L = tab ? load_layer(tab + blockIdx.y) : inl;
  const int tile = blockIdx.x;
  const int64_t K = L.K;
  const bool vec = (reinterpret_cast<uintptr_t>(L.x) & 15) == 0;
  int E[2] = {0, 0};
  if constexpr (MODE == kModeBf16 || MODE == kModeBf16F4) {
    __shared__ float red[4][2];
    __shared__ int sh_E[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int b = 2 * tile + s;
      float m = 0.0f;
      if (b < h.B) {
        const uint16_t* xb = static_cast<const uint16_t*>(L.x) + (int64_t)b * K * 2;
        if (vec) {
          const uint4* xv = reinterpret_cast<const uint4*>(xb);
          for (int64_t i = threadIdx.x; i < K / 4; i += blockDim.x) {  // 8 bf16 (4 complex) per vector
            const uint4 w = xv[i];
            const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int j = 0; j < 4; ++j)
              m = fmaxf(m, fmaxf(fabsf(__uint_as_float(wd[j] << 16)), fabsf(__uint_as_float(wd[j] & 0xFFFF0000u))));
          }
        } else {
          for (int64_t i = threadIdx.x; i < 2 * K; i += blockDim.x)
            m = fmaxf(m, fabsf(__uint_as_float((uint32_t)xb[i] << 16)));
        }
      }
      for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
      if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6][s] = m;
    }
    __syncthreads();
    if (threadIdx.x < 2) {
      const int s = threadIdx.x, b = 2 * tile + s;
      const float g = fmaxf(fmaxf(red[0][s], red[1][s]), fmaxf(red[2][s], red[3][s]));
      int ex = 0, e = 0;
      if (g > 0.0f) {
        frexpf(g, &ex);       // g in [2^(ex-1), 2^ex)
        // g * 2^e in [2^21, 2^22) (3 base-256 digits) or [2^14, 2^15) (4 base-16 digits)
        e = (MODE == kModeBf16 ? 22 : 15) - ex;
        if (e > 149) e = 149; // keep 2^-e representable in float32
      }
      sh_E[s] = e;
      if (b < h.B && blockIdx.z == 0) L.xs[b] = g > 0.0f ? ldexpf(1.0f, -e) : 0.0f;
    }
    __syncthreads();
    E[0] = sh_E[0];
    E[1] = sh_E[1];
  } else {
    if (threadIdx.x < 8 && blockIdx.z == 0) {
      // the accumulator export passes no factors (its epilogue does not use them)
      const int b = 8 * tile + threadIdx.x;
      if (b < h.B) L.xs[b] = L.x_scale_in ? L.x_scale_in[b] : 1.0f;
    }
  }
  const int nch = L.nk4 * 16 * h.nc;
  uint4* dst = reinterpret_cast<uint4*>(L.xf) + (int64_t)tile * nch;
  if constexpr (MODE == kModeBf16F4) {
    // one thread per run of 16 values of one component of one token: it
    // writes the run's four digit chunks (columns 8 tk + 2 digit + comp)
    const int ntok = h.nc / 8;
    const int nrun = L.nk4 * 16 * ntok * 2;
    for (int ri = blockIdx.z * blockDim.x + threadIdx.x; ri < nrun; ri += gridDim.z * blockDim.x) {
      const int comp = ri & 1, tk = (ri >> 1) % ntok, r = (ri >> 1) / ntok;
      const int kk = r >> 4, d = (r >> 2) & 3, g = r & 3;
      const int64_t k0 = (int64_t)kk * 256 + 64 * d + 16 * g;
      const int b = 2 * tile + tk;
      uint32_t out[4][4] = {};
      if (b < h.B && k0 < K) {  // K % 64 == 0: the whole run is in range
        int v[16];
        load_run16<kModeBf16>(L.x, vec, ((int64_t)b * K + k0) * 2, comp, v);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          int X = (int)rintf(ldexpf(__uint_as_float((uint32_t)v[e] << 16), tk ? E[1] : E[0]));
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            // balanced base-16 digits of |X| <= 2^15: d_0..d_2 in [-8, 7], |d_3| <= 9
            const int dj = j < 3 ? ((X + 8) & 15) - 8 : X;
            X = (X - dj) >> 4;
            out[j][e >> 2] |= e4m3_of_int(dj) << (8 * (e & 3));
          }
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j)
        dst[(int64_t)r * h.nc + 8 * tk + 2 * j + comp] = make_uint4(out[j][0], out[j][1], out[j][2], out[j][3]);
    }
    return;
  }
  for (int ch = blockIdx.z * blockDim.x + threadIdx.x; ch < nch; ch += gridDim.z * blockDim.x) {
    const int col = ch % h.nc, r = ch / h.nc;
    const int kk = r >> 4, d = (r >> 2) & 3, g = r & 3;
    const int64_t k0 = (int64_t)kk * 256 + 64 * g + 16 * d;  // chunk (d, g) feeds dword d of lane group g
    uint32_t out[4] = {0u, 0u, 0u, 0u};
    int b, digit, comp;
    if (col_token<MODE>(tile, col, h.B, b, digit, comp) && k0 < K) {  // K % 64 == 0: whole run in range
      int v[16];
      load_run16<MODE>(L.x, vec, ((int64_t)b * K + k0) * 2, comp, v);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int dd = e >> 2, bb = e & 3;  // byte 4dd+bb holds code dd + 4bb of the run
        int q = v[dd + 4 * bb];
        if constexpr (MODE == kModeBf16) {
          const int X = (int)rintf(ldexpf(__uint_as_float((uint32_t)q << 16), (b & 1) ? E[1] : E[0]));
          const int d0 = ((X + 128) & 255) - 128;
          const int X1 = (X - d0) >> 8;
          const int d1 = ((X1 + 128) & 255) - 128;
          const int d2 = (X1 - d1) >> 8;
          q = digit == 0 ? d0 : (digit == 1 ? d1 : d2);
        }
        out[dd] |= ((uint32_t)q & 0xFFu) << (8 * bb);
      }
    }
    dst[ch] = make_uint4(out[0], out[1], out[2], out[3]);
  }
}

// Position of one pass (work item x tile group) inside its layer.
struct PassGeo {
  int rb, kc, tg0, row, k4b, nk4_item;
  bool row_ok;
};

__device__ inline PassGeo pass_geo(const DecLayer& L, int64_t item, int tg0, int li) {
  PassGeo q;
  const int64_t local = item - L.item0;
  q.rb = (int)(local / L.nkc);
  q.kc = (int)(local - (int64_t)q.rb * L.nkc);
  q.tg0 = tg0;
  q.row = q.rb * 16 + li;
  q.row_ok = q.row < L.N;
  q.k4b = q.kc * L.kc4;
  q.nk4_item = min(L.kc4, L.nk4 - q.k4b);
  return q;
}

// Issue the loads of step j of a pass (the 2T code planes' 16 bytes per lane
// and the activation operand of the tile group).  Out-of-range lanes use an
// offset past the buffer and read 0.
template <int MODE, int T, int NTG>
__device__ inline void issue_step_loads(const DecLayer& L, const DecHeader& h, const PassGeo& q, int lane, int j,
                                        v4i (&cw)[2 * T][kRegKc4], v4i (&xa)[kRegKc4][4][NTG]) {
  const int g = lane >> 4, li = lane & 15;
  const int K = L.K;
  const int kk = q.k4b + j;
  const bool kok = j < q.nk4_item;
  const bool ok = q.row_ok && kok && kk * 256 + 64 * g < K;
  if (L.tiled) {
    // tile (rb, kk, t) is one 1024-byte run; this lane's 16 bytes sit at lane * 16
    const uint32_t mat_bytes = (uint32_t)(T * L.nrb * L.nk4 * 1024);
    const uint32_t off = ok ? (uint32_t)((q.rb * L.nk4 + kk) * T) * 1024u + (uint32_t)lane * 16u : kOob;
#pragma unroll
    for (int p = 0; p < 2 * T; ++p) {
      const int m = p / T, t = p % T;
      cw[p][j] = __builtin_amdgcn_raw_buffer_load_b128(make_rsrc(L.codes[m] + t * 1024, mat_bytes - t * 1024), off, 0,
                                                       kNonTemporal);
    }
  } else {
    const uint32_t plane_bytes = (uint32_t)((int64_t)L.N * K / 4);
    const uint32_t off = ok ? (uint32_t)q.row * (uint32_t)(K / 4) + (uint32_t)(kk * 64 + 16 * g) : kOob;
#pragma unroll
    for (int p = 0; p < 2 * T; ++p) {
      const int m = p / T, t = p % T;
      cw[p][j] = __builtin_amdgcn_raw_buffer_load_b128(make_rsrc(L.codes[m] + (int64_t)t * plane_bytes, plane_bytes),
                                                       off, 0, kNonTemporal);
    }
  }
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(L.xf, (uint32_t)(h.ntile * L.nk4 * 256 * h.nc));
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int tt = 0; tt < NTG; ++tt) {
      const int tile = q.tg0 + tt;
      int b, digit, comp;
      const bool ok = kok && tile < h.ntile && col_token<MODE>(tile, li, h.B, b, digit, comp);
      const uint32_t off = ok ? (uint32_t)(((((tile * L.nk4 + kk) * 4 + d) * 4 + g) * h.nc + li) * 16) : kOob;
      xa[j][d][tt] = buf_load16(xr, off);
    }
}

// Factor of this lane's token s (bf16: token 2*tile + g/2; int8: token
// 8*tile + 2g + s) from the tile's preloaded factors, selected with
// compile-time indices only.
template <int MODE>
__device__ inline float token_factor(const float (&xsv)[8], int g, int s) {
  if constexpr (MODE == kModeBf16) {
    return (g >> 1) ? xsv[1] : xsv[0];
  } else {
    const float f0 = s ? xsv[1] : xsv[0], f1 = s ? xsv[3] : xsv[2];
    const float f2 = s ? xsv[5] : xsv[4], f3 = s ? xsv[7] : xsv[6];
    return g == 0 ? f0 : (g == 1 ? f1 : (g == 2 ? f2 : f3));
  }
}

// Epilogue of a pass: lane holds x columns 4g..4g+3 of weight row li for each
// (plane, axis, tile) accumulator; forms y (or the split-K partial, or the
// exported integer products) of its row for the tokens of those columns.
template <int MODE, int T, int NTG, bool EXPORT>
__device__ inline void write_outputs(const DecLayer& L, const DecHeader& h, const PassGeo& q, int lane,
                                     const v4i (&acc)[2 * T][2][NTG]) {
  // no fused multiply-adds: every inlined copy rounds alike, so y does not
  // depend on which wave or ring slot finishes an item
#pragma clang fp contract(off)
  constexpr int P = 2 * T;
  const int g = lane >> 4;
  const int N = L.N;
  // wave-uniform operands of the epilogue, by scalar loads
  float sc[2][T][2];
  if constexpr (!EXPORT) sload_scales<T>(L.scales[0], L.scales[1], sc);
#pragma unroll
  for (int tt = 0; tt < NTG; ++tt) {
    const int tile = q.tg0 + tt;
    // factors of the (up to 8) tokens of this tile
    float xsv[8];
    if constexpr (!EXPORT) {
      // the factor array is padded to 256 bytes, so the tile's full run of
      // nt floats is always inside it
      constexpr int nt = MODE == kModeBf16 ? 2 : 8;
      float run[nt];
      sload_run<nt>(L.xs + tile * nt, run);
#pragma unroll
      for (int i = 0; i < 8; ++i) xsv[i] = (i < nt && tile * nt + i < h.B) ? run[i < nt ? i : 0] : 0.0f;
    }
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
    if (!q.row_ok || tile >= h.ntile) continue;
    const int ntok = MODE == kModeBf16 ? ((g & 1) ? 0 : 1) : 2;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int b = MODE == kModeBf16 ? 2 * tile + (g >> 1) : 8 * tile + 2 * g + s;
      if (s >= ntok || b >= h.B) continue;
      if constexpr (EXPORT) {
#pragma unroll
        for (int p = 0; p < P; ++p)
#pragma unroll
          for (int ax = 0; ax < 2; ++ax) {
            int32_t* dst = L.acc + ((((int64_t)p * 2 + ax) * h.B + b) * N + q.row) * 2;
            atomicAdd(dst, acc[p][ax][tt][2 * s]);
            atomicAdd(dst + 1, acc[p][ax][tt][2 * s + 1]);
          }
      } else {
        // exact integer product of plane (p, ax) with component c of token b,
        // as a double: digits 0 and 1 combine exactly in int32, digit 2 in double
        auto Pv = [&](int p, int ax, int c) -> double {
          if constexpr (MODE == kModeBf16)
            return (double)(acc[p][ax][tt][c] + (acc[p][ax][tt][2 + c] << 8)) + 65536.0 * (double)hi[p][ax][c];
          else
            return (double)acc[p][ax][tt][2 * s + c];
        };
        double yr = 0.0, yi = 0.0;
#pragma unroll
        for (int t = 0; t < T; ++t) {
          const double su_re = sc[0][t][0], su_im = sc[0][t][1];
          const double sw_re = sc[1][t][0], sw_im = sc[1][t][1];
          const int pu = t, pw = T + t;
          yr += su_re * Pv(pu, 0, 0) - su_im * Pv(pu, 1, 1);
          yi += su_re * Pv(pu, 0, 1) + su_im * Pv(pu, 1, 0);
          yr += sw_re * Pv(pw, 0, 0) + sw_im * Pv(pw, 1, 1);
          yi += -sw_re * Pv(pw, 0, 1) + sw_im * Pv(pw, 1, 0);
        }
        const double f = (double)token_factor<MODE>(xsv, g, s);
        const float2 v = make_float2((float)(yr * f), (float)(yi * f));
        // buffer stores: a global-only access, so no wait on in-flight loads into LDS
        if (L.nkc == 1)
          buf_store8(L.y, (uint32_t)h.B * N * 8, (uint32_t)((b * N + q.row) * 8), v);
        else
          buf_store8(L.part, (uint32_t)L.nkc * h.B * N * 8, (uint32_t)(((q.kc * h.B + b) * N + q.row) * 8), v);
      }
    }
  }
}

// Products of one pass and its epilogue.
template <int MODE, int T, int NTG, bool EXPORT>
__device__ inline void compute_pass(const DecLayer& L, const DecHeader& h, const PassGeo& q, int lane,
                                    v4i (&cw)[2 * T][kRegKc4], v4i (&xa)[kRegKc4][4][NTG], bool has_next,
                                    const DecLayer& Ln, const PassGeo& qn) {
  constexpr int P = 2 * T;
  const int g = lane >> 4;
  v4i acc[P][2][NTG];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int ax = 0; ax < 2; ++ax)
#pragma unroll
      for (int tt = 0; tt < NTG; ++tt) acc[p][ax][tt] = v4i{0, 0, 0, 0};

#pragma unroll
  for (int j = 0; j < kRegKc4; ++j) {
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
    // step j's registers are free: start the next pass's step j
    if (has_next) issue_step_loads<MODE, T, NTG>(Ln, h, qn, lane, j, cw, xa);
  }

  write_outputs<MODE, T, NTG, EXPORT>(L, h, q, lane, acc);
}

// Persistent product kernel: wave w owns the contiguous range of passes
// [w P / W, (w+1) P / W) (a pass = one work item and one tile group).  The
// layer descriptor is kept while the range stays in one layer, and the loads
// of the next pass go into each register set as soon as the current pass has
// finished reading it, so they overlap the rest of the pass and its epilogue.
template <int MODE, int T, int NTG, bool EXPORT>
__global__ __launch_bounds__(256) void dec_mfma_kernel(DecHeader h, DecLayer inl,
                                                       const DecLayer* __restrict__ tab) {
  constexpr int P = 2 * T;
  const int lane = threadIdx.x & 63;
  const int li = lane & 15;
  const int64_t wid = (int64_t)blockIdx.x * 4 + uniform(threadIdx.x >> 6);
  const int64_t W = (int64_t)gridDim.x * 4;
  const int ngroups = (h.ntile + NTG - 1) / NTG;
  const int64_t total = h.total_items * ngroups;
  int64_t pass = uniform64(wid * total / W);
  const int64_t pend = uniform64((wid + 1) * total / W);
  if (pass >= pend) return;

  int lidx = tab ? find_layer(tab, h.n_layers, pass / ngroups) : 0;
  DecLayer L = tab ? load_layer(tab + lidx) : inl;
  int64_t lend = L.item0 + (int64_t)L.nrb * L.nkc;  // first item past layer L
  PassGeo q = pass_geo(L, pass / ngroups, (int)(pass % ngroups) * NTG, li);

  v4i cw[P][kRegKc4];
  v4i xa[kRegKc4][4][NTG];
#pragma unroll
  for (int j = 0; j < kRegKc4; ++j) issue_step_loads<MODE, T, NTG>(L, h, q, lane, j, cw, xa);

  while (true) {
    const bool has_next = pass + 1 < pend;
    DecLayer Ln = L;
    int64_t lendn = lend;
    PassGeo qn = q;
    if (has_next) {
      const int64_t it = (pass + 1) / ngroups;
      if (it >= lend) {  // the range crosses into the next layer
        ++lidx;
        Ln = load_layer(tab + lidx);
        lendn = Ln.item0 + (int64_t)Ln.nrb * Ln.nkc;
      }
      qn = pass_geo(Ln, it, (int)((pass + 1) % ngroups) * NTG, li);
    }
    compute_pass<MODE, T, NTG, EXPORT>(L, h, q, lane, cw, xa, has_next, Ln, qn);
    if (!has_next) break;
    pass += 1;
    L = Ln;
    lend = lendn;
    q = qn;
  }
}

// ------------------------------------------------------ streaming kernel ---
// For one activation tile (bf16 B <= 2, int8 B <= 8) each wave streams its
// range of work items through a ring of NS slots, filled NS-1 steps (of 256
// codes) ahead of the step being computed.  A slot holds the step's code
// bytes in registers (16 bytes per lane and plane, non-temporal loads: the
// codes are read once) and its activation operand in LDS (a direct-to-LDS
// load of the layer's prepared operand, which stays cached: every row block
// of the layer reads it).  Out-of-range lanes load zeros.  A lane only ever
// reads its own wave's slots, so waves never wait for each other.  A work
// item spans kc4 steps (up to 2048 codes), which keeps the epilogue cost per
// code small.

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Geometry of one layer as the streaming kernel needs it (all wave-uniform).
struct StreamLayer {
  int64_t item0, lend;  // first work item of the layer and one past its last
  int32_t N, K, nkc, kc4, nk4, tiled;
};

__device__ inline StreamLayer stream_layer(const DecLayer& L) {
  StreamLayer g;
  g.item0 = L.item0;
  g.lend = L.item0 + (int64_t)L.nrb * L.nkc;
  g.N = L.N;
  g.K = L.K;
  g.nkc = L.nkc;
  g.kc4 = L.kc4;
  g.nk4 = L.nk4;
  g.tiled = L.tiled;
  return g;
}

// Load side of the streaming kernel: which step's bytes to fetch next.  All
// geometry is recomputed only when an item starts; a step just advances two
// offsets.  Only addressing state is kept (a layer descriptor is read from
// the table when the range enters a new layer).
template <int T>
struct LoadCursor {
  StreamLayer G;
  int64_t item;
  int lidx, rb, kc, j, nsteps, k4;  // item = (row block rb, K slice kc) of layer lidx
  const uint8_t* pbase[2 * T];  // code plane (M, t) of the current layer
  const int8_t* xf;             // the layer's activation operand
  uint32_t plane_bytes, xbytes;
  uint32_t xtile;  // bytes of one activation tile's operand
  uint32_t voff;   // this lane's offset in every code plane at step k4 (row, 16-code group)
  uint32_t vstep;  // voff advance per step: 64 (D3) or T * 1024 (tiled)
  uint32_t xoff;   // offset of the step's activation operand + lane * 16
  bool row_ok;
};

// (row block, K slice) of an item inside its layer (a layer has < 2^31 items)
__device__ inline void split_item(int64_t item, const StreamLayer& G, int& rb, int& kc) {
  const int local = (int)(item - G.item0);
  rb = local / G.nkc;
  kc = local - rb * G.nkc;
}

// The next item of a cursor: the next K slice, else the next row block.
__device__ inline void advance_item(int& rb, int& kc, int nkc) {
  if (++kc == nkc) {
    kc = 0;
    ++rb;
  }
}

template <int T>
__device__ inline void load_item(LoadCursor<T>& c, const DecHeader& h, int lane) {
  const int g = lane >> 4, li = lane & 15;
  const int rb = c.rb, kc = c.kc;
  c.k4 = kc * c.G.kc4;
  c.nsteps = min(c.G.kc4, c.G.nk4 - c.k4);
  c.j = 0;
  const int row = rb * 16 + li;
  c.row_ok = row < c.G.N;
  c.voff = c.G.tiled ? (uint32_t)((rb * c.G.nk4 + c.k4) * T) * 1024u + (uint32_t)lane * 16u
                     : (uint32_t)row * (uint32_t)(c.G.K / 4) + (uint32_t)(c.k4 * 64 + 16 * g);
  c.xoff = (uint32_t)(c.k4 * 256 * h.nc + lane * 16);
}

template <int T>
__device__ inline void load_enter_layer(LoadCursor<T>& c, const DecLayer& L, const DecHeader& h) {
  c.G = stream_layer(L);
  if (L.tiled) {
    // every stage's tiles are addressed from the matrix base + t * 1024
    c.plane_bytes = (uint32_t)(T * L.nrb * L.nk4 * 1024) - (uint32_t)(T - 1) * 1024u;
#pragma unroll
    for (int p = 0; p < 2 * T; ++p) c.pbase[p] = L.codes[p / T] + (p % T) * 1024;
    c.vstep = (uint32_t)T * 1024u;
  } else {
    c.plane_bytes = (uint32_t)((int64_t)L.N * L.K / 4);
#pragma unroll
    for (int p = 0; p < 2 * T; ++p) c.pbase[p] = L.codes[p / T] + (int64_t)(p % T) * c.plane_bytes;
    c.vstep = 64u;
  }
  c.xf = L.xf;
  c.xtile = (uint32_t)(L.nk4 * 256 * h.nc);
  c.xbytes = (uint32_t)h.ntile * c.xtile;
}

// Issue the loads of the cursor's step: its 2T x 16 code bytes per lane into
// registers cq, and its activation operand (XW KiB for each of NT tiles) into
// the LDS slot xslot.
// A dead cursor issues them out of range (they return zeros), so every step
// issues the same number of loads.  Lane group g's first code of the step is
// code 64 g (D3 and tiled layouts) or 32 g (fp4 tiled layout, G0 = 32); a
// group whose codes all lie past K loads zeros.
template <int XW, int T, int G0 = 64, int NT = 1>
__device__ inline void stream_issue(const LoadCursor<T>& c, bool live, int lane, v4i (&cq)[2 * T],
                                    uint8_t* xslot) {
  const int g = lane >> 4;
  const bool ok = live && c.row_ok && c.k4 * 256 + G0 * g < c.G.K;
  const uint32_t off = ok ? c.voff : kOob;
  // descriptor fields stated wave-uniform, so the descriptors stay in scalar
  // registers (no per-load waterfall over lanes)
  const int pb = __builtin_amdgcn_readfirstlane((int)c.plane_bytes);
#pragma unroll
  for (int p = 0; p < 2 * T; ++p)
    cq[p] = __builtin_amdgcn_raw_buffer_load_b128(make_rsrc(uniform_ptr(c.pbase[p]), (uint32_t)pb), off, 0,
                                                  kNonTemporal);
  const int xb = __builtin_amdgcn_readfirstlane((int)c.xbytes);
  const int8_t* xf = uniform_ptr(c.xf);
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < XW; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(make_rsrc(xf, (uint32_t)xb), (lds_ptr_t)(xslot + (t * XW + i) * 1024),
                                               16, live ? c.xoff + t * c.xtile + i * 1024 : kOob, 0, 0, 0);
}

// LDS address (byte offset) of a pointer into shared memory.
__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)reinterpret_cast<uintptr_t>((lds_ptr_t)const_cast<void*>(p));
}

// Four 16-byte LDS reads and the wait for them, as one unit.  The ring's
// loads into LDS are ordered by the caller's explicit vmcnt wait; written
// this way the compiler adds no wait of its own for the loads still in
// flight into the ring's other slots.
__device__ inline void lds_read4(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3, v4i (&x)[4]) {
  __asm__ volatile(
      "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\tds_read_b128 %3, %7\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(x[0]), "=&v"(x[1]), "=&v"(x[2]), "=&v"(x[3])
      : "v"(a0), "v"(a1), "v"(a2), "v"(a3)
      : "memory");
}

// Compute side: which item the current step belongs to, and what its
// epilogue writes.
struct OutCursor {
  StreamLayer G;
  const float* scales[2];
  float* xs;
  float2* y;
  float2* part;
  int64_t item;
  int lidx, rb, kc, j, nsteps, row;
  bool row_ok;
};

__device__ inline void out_enter_layer(OutCursor& c, const DecLayer& L) {
  c.G = stream_layer(L);
  c.scales[0] = L.scales[0];
  c.scales[1] = L.scales[1];
  c.xs = L.xs;
  c.y = L.y;
  c.part = L.part;
}

__device__ inline void out_item(OutCursor& c, int li) {
  c.nsteps = min(c.G.kc4, c.G.nk4 - c.kc * c.G.kc4);
  c.j = 0;
  c.row = c.rb * 16 + li;
  c.row_ok = c.row < c.G.N;
}

// The fields write_outputs reads, from the compute cursor.
__device__ inline DecLayer out_layer(const OutCursor& c) {
  DecLayer L{};
  L.scales[0] = uniform_ptr(c.scales[0]);
  L.scales[1] = uniform_ptr(c.scales[1]);
  L.xs = uniform_ptr(c.xs);
  L.y = uniform_ptr(c.y);
  L.part = uniform_ptr(c.part);
  L.N = c.G.N;
  L.nkc = c.G.nkc;
  return L;
}

// Items the load cursor has entered and the output cursor has not reached
// (the load side runs at most NS - 1 <= 3 steps ahead, an item has >= 1 step),
// as offsets from the block's first item.
struct ItemQueue {
  int q0, q1, q2, q3;
  int n;
  __device__ void push(int v) {
    if (n == 0) q0 = v;
    else if (n == 1) q1 = v;
    else if (n == 2) q2 = v;
    else q3 = v;
    ++n;
  }
  __device__ int pop() {
    const int v = q0;
    q0 = q1;
    q1 = q2;
    q2 = q3;
    --n;
    return v;
  }
};

// Offset of this wave's next item in its block's range of n items, or -1:
// lane 0 takes a ticket from the block's LDS counter.  Written as one asm
// block so that the compiler adds no wait for the loads still in flight into
// the LDS ring.
__device__ inline int claim_item(uint32_t ctr_addr, int n, int lane) {
  int off = 0;
  if (lane == 0) {
    __asm__ volatile("ds_add_rtn_u32 %0, %1, %2\n\ts_waitcnt lgkmcnt(0)"
                     : "=v"(off)
                     : "v"(ctr_addr), "v"(1)
                     : "memory");
  }
  off = uniform(off);
  return off < n ? off : -1;
}

// Move a cursor to `item` (>= its current item) of the layer table.
template <int T>
__device__ inline void load_goto(LoadCursor<T>& c, int64_t item, const DecLayer* tab, const DecHeader& h,
                                 int lane) {
  while (item >= c.G.lend) {
    ++c.lidx;
    load_enter_layer(c, load_layer(tab + c.lidx), h);
  }
  c.item = item;
  split_item(item, c.G, c.rb, c.kc);
  load_item(c, h, lane);
}

// Returns whether the cursor entered another layer.
__device__ inline bool out_goto(OutCursor& c, int64_t item, const DecLayer* tab, int li) {
  bool moved = false;
  while (item >= c.G.lend) {
    ++c.lidx;
    out_enter_layer(c, load_layer(tab + c.lidx));
    moved = true;
  }
  c.item = item;
  split_item(item, c.G, c.rb, c.kc);
  out_item(c, li);
  return moved;
}

// One block per CU for both streaming kernels: the waves that share a SIMD
// are served in age order, so a static split of the items across them leaves
// the youngest wave of each SIMD working long after the oldest has finished.
// The block's waves therefore claim their items one at a time from a counter
// in LDS.  Three waves per SIMD for T <= 2; two for T >= 3, whose
// accumulators and ring need more than 168 registers.
constexpr int block_waves(int T) { return T <= 2 ? 12 : 8; }

// waves per block of the streaming kernel (fewer when the ring would not
// fit the LDS)
constexpr int kStreamWaves = 4;
constexpr int stream_waves(int NS, int XW, int base = kStreamWaves) {
  int w = base;
  while (w > 1 && w * NS * XW * 1024 > 150 * 1024) w /= 2;
  return w;
}

// ring depth: about 48 code registers per lane
constexpr int ring_slots(int T) { return T <= 1 ? 4 : (T == 2 ? 3 : 2); }

template <int T, int XW, int NSLOTS = ring_slots(T), int BASE_WAVES = block_waves(T)>
struct StreamCfg {
  static constexpr int P = 2 * T;
  static constexpr int XSLOT = XW * 1024;         // LDS bytes of a slot's activation operand
  static constexpr int NS = NSLOTS;
  static constexpr int WAVES = stream_waves(NS, XW, BASE_WAVES);
  static constexpr int LOADS = P + XW;            // vector memory ops issued per step
  static constexpr int WAIT = (NS - 1) * LOADS;   // outstanding ops allowed when a slot is read
  static constexpr int WAITCNT = (WAIT & 0xF) | (0x7 << 4) | (0xF << 8) | (((WAIT >> 4) & 3) << 14);
};

template <int MODE, int T, int XW>
__global__ __launch_bounds__((64 * StreamCfg<T, XW>::WAVES)) void dec_stream_kernel(DecHeader h, DecLayer inl,
                                                                       const DecLayer* __restrict__ tab) {
#if defined(__HIP_DEVICE_COMPILE__)  // LDS-DMA and buffer-descriptor code: device pass only
  using C = StreamCfg<T, XW>;
  constexpr int P = C::P, NS = C::NS, XSLOT = C::XSLOT;
  constexpr int WAVES = C::WAVES;
  static_assert(NS <= 4, "the item queue holds the items of up to NS - 1 steps ahead");
  __shared__ __attribute__((aligned(16))) uint8_t ring[WAVES][NS][XSLOT];
  __shared__ __attribute__((aligned(16))) uint8_t zero16[16];
  __shared__ uint32_t claim_ctr;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, li = lane & 15;
  const int wave = uniform(threadIdx.x >> 6);
  if (threadIdx.x < 4) reinterpret_cast<uint32_t*>(zero16)[threadIdx.x] = 0u;
  if (threadIdx.x == 0) claim_ctr = (uint32_t)WAVES;  // wave w starts with item b0 + w
  __syncthreads();
  // the block's items: an equal share of the call's
  const int64_t b0 = uniform64((int64_t)blockIdx.x * h.total_items / gridDim.x);
  const int nb = uniform((int)(uniform64(((int64_t)blockIdx.x + 1) * h.total_items / gridDim.x) - b0));
  if (wave >= nb) return;
  const int64_t i0 = b0 + wave;
  const uint32_t ctr_addr = lds_addr(&claim_ctr);

  // activation operand: this lane's 16 bytes within a slot (or a zero area)
  int b_, digit_, comp_;
  const bool xvalid = col_token<MODE>(0, li, h.B, b_, digit_, comp_);

  LoadCursor<T> lc;
  OutCursor oc;
  ItemQueue iq;
  iq.n = 0;
  {
    const int lidx = tab ? find_layer(tab, h.n_layers, i0) : 0;
    const DecLayer L0 = tab ? load_layer(tab + lidx) : inl;
    lc.lidx = oc.lidx = lidx;
    lc.item = oc.item = i0;
    load_enter_layer(lc, L0, h);
    out_enter_layer(oc, L0);
    split_item(i0, lc.G, lc.rb, lc.kc);
    oc.rb = lc.rb;
    oc.kc = lc.kc;
  }
  load_item(lc, h, lane);
  out_item(oc, li);

  // as in the fp4 kernel: the load side claims items, the output side follows
  auto load_advance = [&]() -> bool {
    if (++lc.j < lc.nsteps) {
      ++lc.k4;
      lc.voff += lc.vstep;
      lc.xoff += 256 * h.nc;
      return true;
    }
    const int off = claim_item(ctr_addr, nb, lane);
    if (off < 0) return false;
    load_goto(lc, b0 + off, tab, h, lane);
    iq.push(off);
    return true;
  };
  auto out_advance = [&]() -> bool {
    if (++oc.j < oc.nsteps) return true;
    if (iq.n == 0) return false;
    out_goto(oc, b0 + iq.pop(), tab, li);
    return true;
  };

  v4i cq[NS][P];  // code bytes of each ring slot
  bool live = true;
#pragma unroll
  for (int k = 0; k < NS - 1; ++k) {
    stream_issue<XW>(lc, live, lane, cq[k], &ring[wave][k][0]);
    if (live) live = load_advance();
  }

  v4i acc[P][2][1];
#pragma unroll
  for (int p = 0; p < P; ++p) acc[p][0][0] = acc[p][1][0] = v4i{0, 0, 0, 0};

  auto step = [&](auto kconst) -> bool {
    constexpr int K = decltype(kconst)::value;
    constexpr int KN = (K + NS - 1) % NS;  // the slot the previous step consumed
    // refill the slot the previous step consumed, then wait for this one
    stream_issue<XW>(lc, live, lane, cq[KN], &ring[wave][KN][0]);
    if (live) live = load_advance();
    __builtin_amdgcn_s_waitcnt(C::WAITCNT);  // this slot's loads have landed
    v4i xr[4];
    {
      const uint32_t xa = xvalid ? lds_addr(&ring[wave][K][0]) + (uint32_t)((g * h.nc + li) * 16) : lds_addr(zero16);
      const uint32_t xs = xvalid ? (uint32_t)(4 * h.nc * 16) : 0u;
      lds_read4(xa, xa + xs, xa + 2 * xs, xa + 3 * xs, xr);
    }
    const v4i* cr = cq[K];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
#pragma unroll
      for (int p = 0; p < P; ++p) {
        v4i bre, bim;
        expand_codes((uint32_t)cr[p][d], bre, bim);
        acc[p][0][0] = __builtin_amdgcn_mfma_i32_16x16x64_i8(xr[d], bre, acc[p][0][0], 0, 0, 0);
        acc[p][1][0] = __builtin_amdgcn_mfma_i32_16x16x64_i8(xr[d], bim, acc[p][1][0], 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 15, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
    }
    if (oc.j == oc.nsteps - 1) {
      PassGeo q;
      q.rb = 0;
      q.kc = oc.kc;
      q.tg0 = 0;
      q.row = oc.row;
      q.row_ok = oc.row_ok;
      q.k4b = 0;
      q.nk4_item = 0;
      write_outputs<MODE, T, 1, false>(out_layer(oc), h, q, lane, acc);
#pragma unroll
      for (int p = 0; p < P; ++p) acc[p][0][0] = acc[p][1][0] = v4i{0, 0, 0, 0};
    }
    return !out_advance();
  };

  // one pass of the loop body visits every slot once, in ring order
  static_assert(NS >= 2 && NS <= 6, "the ring loop below is unrolled for 2..6 slots");
  while (true) {
    if (step(std::integral_constant<int, 0>{})) break;
    if (step(std::integral_constant<int, 1>{})) break;
    if constexpr (NS > 2) if (step(std::integral_constant<int, 2 % NS>{})) break;
    if constexpr (NS > 3) if (step(std::integral_constant<int, 3 % NS>{})) break;
    if constexpr (NS > 4) if (step(std::integral_constant<int, 4 % NS>{})) break;
    if constexpr (NS > 5) if (step(std::integral_constant<int, 5 % NS>{})) break;
  }
  __builtin_amdgcn_s_waitcnt(0);  // no load may still be writing LDS when the wave ends
#endif
}

// ------------------------------------------- streaming kernel, fp4 codes ---
// The same ring, cursors and work items as above, for codes in the fp4 tiled
// layout and bf16 activations as 4 base-16 digits (e4m3 integers).  With the
// code bits (p, q) = (bit 0, bit 1) of code k, i^k = (1 - 2q)(1 - p) +
// i (1 - 2q) p (Eq. realify-ops: b_re = (1 - 2q)(1 - p), b_im = (1 - 2q) p),
// the kernel contracts two e2m1 operands with v_mfma_f32_16x16x128_f8f6f4:
//     S = 1 - 2q  (every code: +-1)     and     I = (1 - 2q) p  (0 or +-1),
// and forms b_re = S - I in the epilogue.  In the fp4 layout a nibble holds
// the bits of two codes at (q_A, q_B, p_A, p_B) = bits (3, 2, 1, 0), so per
// 32-bit word of 16 codes
//     I_A = w & 0xAAAAAAAA,          S_A = I_A | 0x22222222,
//     I_B = (w << 1) & 0xAAAAAAAA,   S_B = I_B | 0x22222222
// (e2m1 0b0010 = 1, 0b1010 = -1, 0b0000 / 0b1000 = +-0): five VALU
// instructions per 16 codes.  Every product is a digit (|d| <= 9) times 0 or
// +-1, so the float32 sums are exact integers (|sum| < 2^24 for K < 2^20).

// S and I operands of one 128-code MFMA from the lane's two code words
// (S = I | 0x22222222: I keeps only bits 3 and 1 of each nibble).
__device__ inline void expand_f4(uint32_t w0, uint32_t w1, v8i& bs, v8i& bi) {
  const uint32_t ia0 = w0 & 0xAAAAAAAAu, ib0 = (w0 << 1) & 0xAAAAAAAAu;
  const uint32_t ia1 = w1 & 0xAAAAAAAAu, ib1 = (w1 << 1) & 0xAAAAAAAAu;
  bi = v8i{(int)ia0, (int)ib0, (int)ia1, (int)ib1, 0, 0, 0, 0};
  bs = v8i{(int)(ia0 | 0x22222222u), (int)(ib0 | 0x22222222u), (int)(ia1 | 0x22222222u),
           (int)(ib1 | 0x22222222u), 0, 0, 0, 0};
}

constexpr int kFmtFp8 = 0;  // MFMA operand format codes: e4m3
constexpr int kFmtFp4 = 4;  // e2m1

// Epilogue of a work item: lane (g, li) holds activation columns 4g..4g+3
// of weight row li, i.e. digits 2(g % 2), 2(g % 2) + 1 of both components of
// token g / 2.  Each lane first joins its two digits (the sums are exact
// integers: an item spans at most 2048 codes, so |sum| < 2^26); odd lane
// groups pass theirs to the even group below, which forms the token's
// integer products and applies the axis scales and the token factor in
// float32.
// The layer's axis scales sc[m][t][axis] and token factors xf[b] are the
// caller's (loaded once per layer).
template <int T>
__device__ inline void write_outputs_f4(const DecLayer& L, const DecHeader& h, int kc, int row, bool row_ok,
                                        int lane, int tile, const v4f (&aS)[2 * T], const v4f (&aI)[2 * T],
                                        const float (&sc)[2][T][2], const float (&xf)[2]) {
  constexpr int P = 2 * T;
  const int g = lane >> 4;
  int vS[P][2], vI[P][2], hS[P][2], hI[P][2];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      vS[p][c] = (int)aS[p][c] + 16 * (int)aS[p][2 + c];
      vI[p][c] = (int)aI[p][c] + 16 * (int)aI[p][2 + c];
      hS[p][c] = __shfl_down(vS[p][c], 16);
      hI[p][c] = __shfl_down(vI[p][c], 16);
    }
  const int b = 2 * tile + (g >> 1);
  if ((g & 1) || !row_ok || b >= h.B) return;
  float yr = 0.0f, yi = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    float Pre[2][2], Pim[2][2];  // [matrix][component]: products with b_re = S - I and b_im = I
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const int p = m * T + t;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const int ii = vI[p][c] + 256 * hI[p][c];
        Pre[m][c] = (float)(vS[p][c] + 256 * hS[p][c] - ii);
        Pim[m][c] = (float)ii;
      }
    }
    // explicit fused multiply-adds in a fixed order: every inlined copy of
    // this epilogue rounds alike, so y does not depend on which wave or ring
    // slot finishes the item
    const float su_re = sc[0][t][0], su_im = sc[0][t][1];
    const float sw_re = sc[1][t][0], sw_im = sc[1][t][1];
    yr = fmaf(su_re, Pre[0][0], yr);
    yr = fmaf(-su_im, Pim[0][1], yr);
    yr = fmaf(sw_re, Pre[1][0], yr);
    yr = fmaf(sw_im, Pim[1][1], yr);
    yi = fmaf(su_re, Pre[0][1], yi);
    yi = fmaf(su_im, Pim[0][0], yi);
    yi = fmaf(-sw_re, Pre[1][1], yi);
    yi = fmaf(sw_im, Pim[1][0], yi);
  }
  const float f = (g >> 1) ? xf[1] : xf[0];
  const float2 v = make_float2(__fmul_rn(yr, f), __fmul_rn(yi, f));
  if (L.nkc == 1)
    buf_store8(L.y, (uint32_t)h.B * L.N * 8, (uint32_t)((b * L.N + row) * 8), v);
  else
    buf_store8(L.part, (uint32_t)L.nkc * h.B * L.N * 8, (uint32_t)(((kc * h.B + b) * L.N + row) * 8), v);
}

constexpr int f4_ring_slots(int T) { return ring_slots(T); }


template <int T, int XW>
using F4Cfg = StreamCfg<T, XW, f4_ring_slots(T), block_waves(T)>;

// NT activation tiles (2 tokens each); a ring slot holds XW KiB per tile.
template <int T, int XW, int NT>
__global__ __launch_bounds__((64 * F4Cfg<T, NT * XW>::WAVES)) void dec_stream_f4_kernel(DecHeader h, DecLayer inl,
                                                                                       const DecLayer* __restrict__ tab) {
#if defined(__HIP_DEVICE_COMPILE__)  // LDS-DMA and buffer-descriptor code: device pass only
  using C = F4Cfg<T, NT * XW>;
  constexpr int P = C::P, NS = C::NS, XSLOT = C::XSLOT;
  constexpr int WAVES = C::WAVES;
  static_assert(NS <= 4, "the item queue holds the items of up to NS - 1 steps ahead");
  __shared__ __attribute__((aligned(16))) uint8_t ring[WAVES][NS][XSLOT];
  __shared__ __attribute__((aligned(16))) uint8_t zero16[16];
  __shared__ uint32_t claim_ctr;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, li = lane & 15;
  const int wave = uniform(threadIdx.x >> 6);
  if (threadIdx.x < 4) reinterpret_cast<uint32_t*>(zero16)[threadIdx.x] = 0u;
  if (threadIdx.x == 0) claim_ctr = (uint32_t)WAVES;  // wave w starts with item b0 + w
  __syncthreads();
  // the block's items: an equal share of the call's
  const int64_t b0 = uniform64((int64_t)blockIdx.x * h.total_items / gridDim.x);
  const int nb = uniform((int)(uniform64(((int64_t)blockIdx.x + 1) * h.total_items / gridDim.x) - b0));
  if (wave >= nb) return;
  const int64_t i0 = b0 + wave;
  const uint32_t ctr_addr = lds_addr(&claim_ctr);

  bool xvalid[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    int b_, digit_, comp_;
    xvalid[t] = col_token<kModeBf16F4>(t, li, h.B, b_, digit_, comp_);
  }

  LoadCursor<T> lc;
  OutCursor oc;
  ItemQueue iq;
  iq.n = 0;
  {
    const int lidx = tab ? find_layer(tab, h.n_layers, i0) : 0;
    const DecLayer L0 = tab ? load_layer(tab + lidx) : inl;
    lc.lidx = oc.lidx = lidx;
    lc.item = oc.item = i0;
    load_enter_layer(lc, L0, h);
    out_enter_layer(oc, L0);
    split_item(i0, lc.G, lc.rb, lc.kc);
    oc.rb = lc.rb;
    oc.kc = lc.kc;
  }
  load_item(lc, h, lane);
  out_item(oc, li);
  // the epilogue's per-layer constants, reloaded when the output side changes layer
  float esc[2][T][2], exf[NT][2];
  auto load_epilogue_consts = [&]() {
    sload_scales<T>(uniform_ptr(oc.scales[0]), uniform_ptr(oc.scales[1]), esc);
    // the factor array is padded to 256 bytes: both floats of every tile are inside it
#pragma unroll
    for (int t = 0; t < NT; ++t) sload_run<2>(uniform_ptr(oc.xs) + 2 * t, exf[t]);
  };
  load_epilogue_consts();

  // next step of the load side: the next step of its item, else a claimed
  // item (queued for the output side); false once the block's items are gone
  auto load_advance = [&]() -> bool {
    if (++lc.j < lc.nsteps) {
      ++lc.k4;
      lc.voff += lc.vstep;
      lc.xoff += 256 * h.nc;
      return true;
    }
    const int off = claim_item(ctr_addr, nb, lane);
    if (off < 0) return false;
    load_goto(lc, b0 + off, tab, h, lane);
    iq.push(off);
    return true;
  };
  auto out_advance = [&]() -> bool {
    if (++oc.j < oc.nsteps) return true;
    if (iq.n == 0) return false;
    if (out_goto(oc, b0 + iq.pop(), tab, li)) load_epilogue_consts();
    return true;
  };

  v4i cq[NS][P];
  bool live = true;
#pragma unroll
  for (int k = 0; k < NS - 1; ++k) {
    stream_issue<XW, T, 32, NT>(lc, live, lane, cq[k], &ring[wave][k][0]);
    if (live) live = load_advance();
  }

  v4f aS[NT][P], aI[NT][P];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int p = 0; p < P; ++p) aS[t][p] = aI[t][p] = v4f{0.f, 0.f, 0.f, 0.f};

  auto step = [&](auto kconst) -> bool {
    constexpr int K = decltype(kconst)::value;
    constexpr int KN = (K + NS - 1) % NS;
    stream_issue<XW, T, 32, NT>(lc, live, lane, cq[KN], &ring[wave][KN][0]);
    if (live) live = load_advance();
    __builtin_amdgcn_s_waitcnt(C::WAITCNT);
    v4i xr[NT][4];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const uint32_t xa = xvalid[t] ? lds_addr(&ring[wave][K][t * XW * 1024]) + (uint32_t)((g * h.nc + li) * 16)
                                    : lds_addr(zero16);
      const uint32_t xs = xvalid[t] ? (uint32_t)(4 * h.nc * 16) : 0u;
      lds_read4(xa, xa + xs, xa + 2 * xs, xa + 3 * xs, xr[t]);
    }
    const v4i* cr = cq[K];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int p = 0; p < P; ++p) {
        v8i bs, bi;
        expand_f4((uint32_t)cr[p][2 * kb], (uint32_t)cr[p][2 * kb + 1], bs, bi);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const v4i x0 = xr[t][2 * kb], x1 = xr[t][2 * kb + 1];
          const v8i a = v8i{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
          aS[t][p] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bs, aS[t][p], kFmtFp8, kFmtFp4, 0, 0, 0, 0);
          aI[t][p] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bi, aI[t][p], kFmtFp8, kFmtFp4, 0, 0, 0, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NT, 0);
      }
    }
    if (oc.j == oc.nsteps - 1) {
      const DecLayer Lo = out_layer(oc);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        write_outputs_f4<T>(Lo, h, oc.kc, oc.row, oc.row_ok, lane, t, aS[t], aI[t], esc, exf[t]);
#pragma unroll
        for (int p = 0; p < P; ++p) aS[t][p] = aI[t][p] = v4f{0.f, 0.f, 0.f, 0.f};
      }
    }
    return !out_advance();
  };

  static_assert(NS >= 2 && NS <= 6, "the ring loop below is unrolled for 2..6 slots");
  while (true) {
    if (step(std::integral_constant<int, 0>{})) break;
    if (step(std::integral_constant<int, 1>{})) break;
    if constexpr (NS > 2) if (step(std::integral_constant<int, 2 % NS>{})) break;
    if constexpr (NS > 3) if (step(std::integral_constant<int, 3 % NS>{})) break;
    if constexpr (NS > 4) if (step(std::integral_constant<int, 4 % NS>{})) break;
    if constexpr (NS > 5) if (step(std::integral_constant<int, 5 % NS>{})) break;
  }
  __builtin_amdgcn_s_waitcnt(0);  // no load may still be writing LDS when the wave ends
#endif
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

// Blocks of kernel k that fit on the current device at once.
int resident_blocks(const void* k, int threads) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, threads, 0) != hipSuccess || per_cu < 1)
    return 1024;
  return cus * per_cu;
}

template <int MODE, int T, int NTG, bool EXPORT>
void launch_dec(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, int64_t want_blocks,
                hipStream_t s) {
  auto k = dec_mfma_kernel<MODE, T, NTG, EXPORT>;
  static const int resident = resident_blocks(reinterpret_cast<const void*>(k), 256);  // one query per variant
  const int64_t blocks = want_blocks < resident ? want_blocks : resident;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(256), 0, s, h, inl, tab);
}

template <int MODE, bool EXPORT>
void launch_dec_mode(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, int64_t blocks,
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

template <int MODE, int T, int XW>
void launch_stream(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, int64_t want_blocks,
                   hipStream_t s) {
  auto k = dec_stream_kernel<MODE, T, XW>;
  constexpr int waves = StreamCfg<T, XW>::WAVES;
  constexpr int threads = 64 * waves;
  static const int resident = resident_blocks(reinterpret_cast<const void*>(k), threads);
  const int64_t want = (h.total_items + waves - 1) / waves;
  const int64_t blocks = want < resident ? want : resident;
  (void)want_blocks;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), 0, s, h, inl, tab);
}

template <int T, int XW, int NT>
void launch_stream_f4(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s) {
  auto k = dec_stream_f4_kernel<T, XW, NT>;
  constexpr int waves = F4Cfg<T, NT * XW>::WAVES;
  constexpr int threads = 64 * waves;
  static const int resident = resident_blocks(reinterpret_cast<const void*>(k), threads);
  const int64_t want = (h.total_items + waves - 1) / waves;
  const int64_t blocks = want < resident ? want : resident;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), 0, s, h, inl, tab);
}

template <int T>
void launch_stream_f4_t(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s) {
  if (h.ntile >= 2) launch_stream_f4<T, 4, 2>(h, inl, tab, s);  // 3-4 tokens: two tiles
  else if (h.nc <= 8) launch_stream_f4<T, 2, 1>(h, inl, tab, s);  // one token: 8 columns, 2 KB per step
  else launch_stream_f4<T, 4, 1>(h, inl, tab, s);
}

template <int MODE, int T>
void launch_stream_t(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, int64_t blocks,
                     hipStream_t s) {
  const int xw = (h.nc + 3) / 4;  // KB of activation operand per step
  if (xw <= 1) launch_stream<MODE, T, 1>(h, inl, tab, blocks, s);
  else if (xw == 2) launch_stream<MODE, T, 2>(h, inl, tab, blocks, s);
  else launch_stream<MODE, T, 4>(h, inl, tab, blocks, s);
}

template <int MODE>
void launch_stream_mode(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, int64_t blocks,
                        hipStream_t s) {
  switch (h.T) {
    case 1: launch_stream_t<MODE, 1>(h, inl, tab, blocks, s); break;
    case 2: launch_stream_t<MODE, 2>(h, inl, tab, blocks, s); break;
    case 3: launch_stream_t<MODE, 3>(h, inl, tab, blocks, s); break;
    default: launch_stream_t<MODE, 4>(h, inl, tab, blocks, s); break;
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
    hipLaunchKernelGGL(dec_prep_kernel<kModeBf16>, dim3(h.ntile, nl, kPrepSplit), dim3(256), 0, s, h, inl, tab);
  else if (h.mode == kModeBf16F4)
    hipLaunchKernelGGL(dec_prep_kernel<kModeBf16F4>, dim3(h.ntile, nl, kPrepSplit), dim3(256), 0, s, h, inl,
                       tab);
  else
    hipLaunchKernelGGL(dec_prep_kernel<kModeI8>, dim3(h.ntile, nl, kPrepSplit), dim3(256), 0, s, h, inl, tab);
  if ((e = hipGetLastError()) != hipSuccess || (e = mark(1)) != hipSuccess) return e;
  if (export_acc) {
    hipLaunchKernelGGL(fill_i32_kernel, dim3(1024), dim3(256), 0, s, acc, acc_elems);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // 2. products
  const int64_t blocks = (h.total_items + 3) / 4;  // capped at what fits on the device
  if (h.mode == kModeBf16F4) {
    // one or two activation tiles (B <= 4), codes in the fp4 tiled layout: checked by the host code
    switch (h.T) {
      case 1: launch_stream_f4_t<1>(h, inl, tab, s); break;
      case 2: launch_stream_f4_t<2>(h, inl, tab, s); break;
      case 3: launch_stream_f4_t<3>(h, inl, tab, s); break;
      default: launch_stream_f4_t<4>(h, inl, tab, s); break;
    }
  } else if (h.kernel == kKernelStream) {
    if (h.mode == kModeBf16) launch_stream_mode<kModeBf16>(h, inl, tab, blocks, s);
    else launch_stream_mode<kModeI8>(h, inl, tab, blocks, s);
  } else if (h.mode == kModeBf16) {
    launch_dec_mode<kModeBf16, false>(h, inl, tab, blocks, s);
  } else if (export_acc) {
    launch_dec_mode<kModeI8, true>(h, inl, tab, blocks, s);
  } else {
    launch_dec_mode<kModeI8, false>(h, inl, tab, blocks, s);
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

int dec_ntile(int mode, int64_t B) { return mode == kModeI8 ? (int)((B + 7) / 8) : (int)((B + 1) / 2); }

int dec_ncols(int mode, int64_t B) {
  if (mode == kModeBf16) return B >= 2 ? 14 : 6;  // per token 6 digit columns, 8-column stride
  if (mode == kModeBf16F4) return B >= 2 ? 16 : 8;  // per token 8 digit columns
  return B >= 8 ? 16 : (int)(2 * B);
}

DecHeader dec_header(int T, int mode, int64_t B, bool export_acc) {
  DecHeader h{};
  h.T = T;
  h.mode = mode;
  h.B = (int32_t)B;
  h.ntile = dec_ntile(mode, B);
  h.nc = dec_ncols(mode, B);
  h.kernel = (!export_acc && h.ntile == 1) ? kKernelStream : kKernelReg;
  return h;
}

size_t dec_layer_setup(DecLayer& l, const DecHeader& h, bool single, char* ws) {
  l.nrb = (int32_t)((l.N + 15) / 16);
  l.nk4 = (int32_t)((l.K + 255) / 256);
  if (h.kernel == kKernelReg) {
    l.kc4 = kRegKc4;
  } else {
    // slices of up to 8 steps (2048 codes); a single layer gets smaller
    // slices while that is needed to give the GPU ~2048 work items
    l.kc4 = 8;
    if (single)
      while (l.kc4 > 1 && (int64_t)l.nrb * ((l.nk4 + l.kc4 - 1) / l.kc4) < 2048) l.kc4 /= 2;
  }
  l.nkc = (l.nk4 + l.kc4 - 1) / l.kc4;
  const size_t xf_bytes = align256((size_t)h.ntile * l.nk4 * 256 * h.nc);
  const size_t xs_bytes = align256((size_t)h.B * sizeof(float));
  const size_t part_bytes = l.nkc > 1 ? align256((size_t)l.nkc * h.B * l.N * sizeof(float2)) : 0;
  if (ws) {
    l.xf = reinterpret_cast<int8_t*>(ws);
    l.xs = reinterpret_cast<float*>(ws + xf_bytes);
    l.part = part_bytes ? reinterpret_cast<float2*>(ws + xf_bytes + xs_bytes) : nullptr;
  }
  return xf_bytes + xs_bytes + part_bytes;
}

}  // namespace fairy2i
