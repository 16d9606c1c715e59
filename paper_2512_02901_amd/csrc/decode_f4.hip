// Decode product (1..8 tokens) on the fp8 x fp4 matrix cores, for bf16
// activations and codes in the fp4 tiled layout.  Sec. 3.4 / Algorithm 1 with
// the dequantisation of Eq. (ifairy-dequant) and the W conj(x) term of
// Eq. (widely-linear); the codes enter the matrix cores as e2m1 values masked
// straight out of their packed words, the activations as e4m3 digits.
#include "common.h"
#include "decode_dev.h"
#include "f4_operand.h"

namespace fairy2i {

namespace {

// ------------------------------------------------- prep, fp4 code path ---
// Activation operand of the fp8 x fp4 product: see f4_operand.h (token
// shift, two-band / one-band e4m3 digit pairs, operand layout).
constexpr int kPrepF4Threads = 512;
constexpr int kPrepUnroll = 4;     // loads a prep thread issues before using them
constexpr int kPrepF4Blocks = 4;   // blocks per layer (tiles x K slices): each slice finds the token maxima itself
constexpr int kTokensPerTile = 2;      // two bands: 8 operand columns per token
constexpr int kMaxTokensPerTile = 4;   // one band: 4 operand columns per token

// One block per (activation tile, layer): the largest magnitude of each of
// the tile's tokens, then the digits of every value.
__global__ __launch_bounds__(kPrepF4Threads) void dec_prep_f4_kernel(DecHeader h, DecLayer inl,
                                                                     const DecLayer* __restrict__ tab) {
  const DecLayer L = tab ? load_layer(tab + blockIdx.y) : inl;
  // the cooperative product kernel's claim counter starts every call at zero
  if (h.coop_ctr && blockIdx.x == 0 && blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0) *h.coop_ctr = 0u;
  const int tile = blockIdx.x;
  const int K = L.K;
  const int bands = h.bands;
  const int cpt = 4 * bands;        // operand columns per token
  const int tpt = 16 / cpt;         // token slots per 16-column tile
  const int ntok = h.nc / cpt;      // token slots written per tile
  const bool vec = (reinterpret_cast<uintptr_t>(L.x) & 15) == 0;
  __shared__ float red[kPrepF4Threads / 64][kMaxTokensPerTile];
  __shared__ int sh_S[kMaxTokensPerTile];
  const int wave = threadIdx.x >> 6;
  // every thread issues all its loads of a round before reducing them
  constexpr int U = kPrepUnroll;
  for (int tk = 0; tk < tpt; ++tk) {
    const int b = tpt * tile + tk;
    float m = 0.0f;
    if (tk < ntok && b < h.B) {
      const uint16_t* xb = static_cast<const uint16_t*>(L.x) + (int64_t)b * K * 2;
      if (vec) {
        const uint4* xv = reinterpret_cast<const uint4*>(xb);
        for (int i0 = 0; i0 < K / 4; i0 += U * kPrepF4Threads) {  // 8 bf16 (4 complex) per vector
          uint4 w[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const int i = i0 + u * kPrepF4Threads + threadIdx.x;
            w[u] = i < K / 4 ? xv[i] : make_uint4(0u, 0u, 0u, 0u);
          }
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const uint32_t wd[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
#pragma unroll
            for (int j = 0; j < 4; ++j)
              m = fmaxf(m, fmaxf(fabsf(__uint_as_float(wd[j] << 16)), fabsf(__uint_as_float(wd[j] & 0xFFFF0000u))));
          }
        }
      } else {
        for (int i = threadIdx.x; i < 2 * K; i += blockDim.x) m = fmaxf(m, fabsf(__uint_as_float((uint32_t)xb[i] << 16)));
      }
    }
    for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    if ((threadIdx.x & 63) == 0) red[wave][tk] = m;
  }
  __syncthreads();
  if (threadIdx.x < tpt) {
    const int tk = threadIdx.x, b = tpt * tile + tk;
    float g = 0.0f;
    for (int w = 0; w < kPrepF4Threads / 64; ++w) g = fmaxf(g, red[w][tk]);
    const int S = f4_token_shift(g);
    sh_S[tk] = S;
    if (blockIdx.z == 0 && tk < ntok && b < h.B) L.xs[b] = g > 0.0f ? ldexpf(1.0f, -S) : 0.0f;
  }
  __syncthreads();
  // one thread per (16-code run, token, component, half run): 8 values, whose
  // four digit bytes per band go to the halves of the run's 16-byte chunks
  const int nrun = L.nk4 * 16;  // run r holds codes 16 r .. 16 r + 15 (= 256 step + 64 d + 16 g for r = 16 step + 4 d + g)
  uint8_t* dst = reinterpret_cast<uint8_t*>(L.xf) + (int64_t)tile * nrun * h.nc * 16;
  // this block's share of the (run, token, component, half) units: the K
  // range is split over gridDim.z blocks (each finds the token maxima itself)
  const int total = nrun * ntok * 4;
  const int per = (total + (int)gridDim.z - 1) / (int)gridDim.z;
  const int ulo = (int)blockIdx.z * per;
  const int uhi = ulo + per < total ? ulo + per : total;
  for (int idx0 = ulo; idx0 < uhi; idx0 += U * kPrepF4Threads) {
    // the loads of all U units of this thread first, then their digits
    uint32_t wu[U][8];  // (re, im) bf16 pairs of each unit's 8 complex values
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int idx = idx0 + u * kPrepF4Threads + threadIdx.x;
      const int hf = idx & 1, tk = (idx >> 2) % ntok, r = (idx >> 2) / ntok;
      const int b = tpt * tile + tk, k0 = 16 * r + 8 * hf;
#pragma unroll
      for (int e = 0; e < 8; ++e) wu[u][e] = 0u;
      if (idx < uhi && b < h.B && k0 < K) {  // K % 64 == 0: the whole half run is in range
        const uint16_t* p = static_cast<const uint16_t*>(L.x) + ((int64_t)b * K + k0) * 2;
        if (vec) {
          const uint4 v0 = reinterpret_cast<const uint4*>(p)[0], v1 = reinterpret_cast<const uint4*>(p)[1];
          wu[u][0] = v0.x; wu[u][1] = v0.y; wu[u][2] = v0.z; wu[u][3] = v0.w;
          wu[u][4] = v1.x; wu[u][5] = v1.y; wu[u][6] = v1.z; wu[u][7] = v1.w;
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) wu[u][e] = (uint32_t)p[2 * e] | ((uint32_t)p[2 * e + 1] << 16);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int idx = idx0 + u * kPrepF4Threads + threadIdx.x;
      if (idx >= uhi) break;
      const int hf = idx & 1, c = (idx >> 1) & 1, tk = (idx >> 2) % ntok, r = (idx >> 2) / ntok;
      uint32_t out[2][2][2] = {};  // [band][hi, lo][word]: bytes e = 0..7 of the half chunk
      float xv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) xv[e] = __uint_as_float(c ? (wu[u][e] & 0xFFFF0000u) : (wu[u][e] << 16));
      f4_unit_digits(xv, sh_S[tk], bands, out);
      // column cpt tk + 4 band + 2 digit + c of run r; this half is bytes 8 hf .. 8 hf + 7 of its chunk
      f4_store_unit(dst, r, h.nc, cpt * tk, c, hf, bands, out);
    }
  }
}

// Up to four tokens with two bands (one 8-column tile for one token, else
// 16-column tiles of two): one block per layer and token slot reads the token
// once into LDS (E entries per thread, K <= E kPrepF4Threads), reduces its
// largest magnitude and writes its 8 digit columns from LDS: one round of
// loads where the general kernel above takes two.  A slot past the last
// token writes zero digits, as the general kernel does.
template <int E>
__global__ __launch_bounds__(kPrepF4Threads) void dec_prep_f4_token_kernel(DecHeader h, DecLayer inl,
                                                                           const DecLayer* __restrict__ tab) {
  const DecLayer L = tab ? load_layer(tab + blockIdx.x) : inl;
  const int b = blockIdx.y;  // the token slot: tile b / 2, columns 8 (b % 2) .. +7 of 16 (8 columns for one token)
  const bool live = b < h.B;
  if (h.coop_ctr && blockIdx.x == 0 && b == 0 && threadIdx.x == 0) *h.coop_ctr = 0u;
  __shared__ __attribute__((aligned(16))) uint32_t tokw[E * kPrepF4Threads];
  __shared__ float red[kPrepF4Threads / 64];
  __shared__ float sh_g;
  const int K = L.K, tid = threadIdx.x, wave = tid >> 6;
  const bool al4 = (reinterpret_cast<uintptr_t>(L.x) & 3) == 0;
  const uint32_t* x32 = static_cast<const uint32_t*>(L.x) + (int64_t)b * K;
  const uint16_t* x16 = static_cast<const uint16_t*>(L.x) + (int64_t)b * 2 * K;
  uint32_t w[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = tid + e * kPrepF4Threads;
    w[e] = 0u;
    if (live && i < K) w[e] = al4 ? x32[i] : ((uint32_t)x16[2 * i] | ((uint32_t)x16[2 * i + 1] << 16));
  }
  float m = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int i = tid + e * kPrepF4Threads;
    if (i < K) {
      tokw[i] = w[e];
      m = fmaxf(m, fmaxf(fabsf(__uint_as_float(w[e] << 16)), fabsf(__uint_as_float(w[e] & 0xFFFF0000u))));
    }
  }
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((tid & 63) == 0) red[wave] = m;
  __syncthreads();
  if (tid == 0) {
    float g = 0.0f;
    for (int v = 0; v < kPrepF4Threads / 64; ++v) g = fmaxf(g, red[v]);
    sh_g = g;
  }
  __syncthreads();
  const float g = sh_g;
  const int S = f4_token_shift(g);
  if (tid == 0 && live) L.xs[b] = g > 0.0f ? ldexpf(1.0f, -S) : 0.0f;
  uint8_t* const dst[1] = {reinterpret_cast<uint8_t*>(L.xf) + (int64_t)(b >> 1) * L.nk4 * 16 * h.nc * 16};
  f4_encode_token<kPrepF4Threads, 1>(tokw, K, S, L.nk4, dst, 1, h.nc, h.nc == 8 ? 0 : 8 * (b & 1));
}

// ------------------------------------------- streaming kernel, fp4 codes ---
// The same ring, cursors and work items as above, for codes in the fp4 tiled
// layout and bf16 activations as two e4m3 digits per value (hi, lo; see the
// fp4 prep kernel above), two tokens per 16-column tile.  With the
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
// instructions per 16 codes.  Every product is an e4m3 digit times 0 or +-1,
// so the products are exact; the matrix core adds them into the float32
// accumulators.

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

// Token factor tt of a tile's NF factors, selected without indexing a
// register array by a lane-dependent value (such an array lives in scratch
// memory, whose loads share the vector-memory queue with the code loads in
// flight, so a wait for one waits for all).  The factors pass through
// readfirstlane so that the selects choose between values, not between
// loads, which the compiler would otherwise fold back into one indexed load.
template <int NF>
__device__ inline float pick_factor(const float (&xf)[NF], int tt) {
  auto val = [](float x) { return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x))); };
  float f = val(xf[0]);
#pragma unroll
  for (int i = 1; i < NF; ++i) f = tt == i ? val(xf[i]) : f;
  return f;
}

// Epilogue of a work item: lane (g, li) holds activation columns 4g..4g+3
// of weight row li, i.e. (hi re, hi im, lo re, lo im) of band g % 2 of token
// g / 2 of the tile, for every (plane, S or I) accumulator.  Each lane joins
// its band's digits (hi + 2^-5 lo); the odd lane group passes its second band
// down to the even group, which adds it times 2^-8, forms b_re = S - I and
// b_im = I and applies the axis scales and the token factor, all in float32
// with explicit fused multiply-adds in a fixed order: every inlined copy
// rounds alike, so y does not depend on which wave or ring slot finishes the
// item.  The layer's axis scales sc[m][t][axis] and the tile's token factors
// xf[2] are the caller's (loaded once per layer).
// With one band (BANDS = 1) lane group g holds token g of the tile, and
// there is no second band to pass down.
template <int T, int BANDS>
__device__ inline void write_outputs_f4(const DecLayer& L, const DecHeader& h, int kc, int row, bool row_ok,
                                        int lane, int tile, const v4f (&aS)[2 * T], const v4f (&aI)[2 * T],
                                        const float (&sc)[2][T][2], const float (&xf)[4 / BANDS]) {
  constexpr int P = 2 * T;
  const int g = lane >> 4;
  float vS[P][2], vI[P][2];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      vS[p][c] = fmaf(aS[p][2 + c], 1.0f / kLoScale, aS[p][c]);
      vI[p][c] = fmaf(aI[p][2 + c], 1.0f / kLoScale, aI[p][c]);
      if constexpr (BANDS == 2) {
        const float hS = __shfl_down(vS[p][c], 16), hI = __shfl_down(vI[p][c], 16);
        vS[p][c] = fmaf(hS, 1.0f / kBand2Scale, vS[p][c]);
        vI[p][c] = fmaf(hI, 1.0f / kBand2Scale, vI[p][c]);
      }
    }
  const int tt = BANDS == 2 ? g >> 1 : g;  // token slot within the tile
  const int b = (4 / BANDS) * tile + tt;
  if ((BANDS == 2 && (g & 1)) || !row_ok || b >= h.B) return;
  float yr = 0.0f, yi = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    float Pre[2][2], Pim[2][2];  // [matrix][component]: products with b_re = S - I and b_im = I
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const int p = m * T + t;
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        Pre[m][c] = vS[p][c] - vI[p][c];
        Pim[m][c] = vI[p][c];
      }
    }
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
  const float f = pick_factor<4 / BANDS>(xf, tt);
  const float2 v = make_float2(__fmul_rn(yr, f), __fmul_rn(yi, f));
  if (L.nkc == 1)
    buf_store8(L.y, (uint32_t)h.B * L.N * 8, (uint32_t)((b * L.N + row) * 8), v);
  else
    buf_store8(L.part, (uint32_t)L.nkc * h.B * L.N * 8, (uint32_t)(((kc * h.B + b) * L.N + row) * 8), v);
}

// Split planes (one-band tiles): the half of write_outputs_f4's sum that
// matrix m (0: U with x, 1: W with conj(x)) contributes, stages in order,
// without the token factor.
template <int T>
__device__ inline float2 partial_outputs_f4(int m, const v4f (&aS)[T], const v4f (&aI)[T], const float (&sc)[2][T][2]) {
  float yr = 0.0f, yi = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    float vS[2], vI[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      vS[c] = fmaf(aS[t][2 + c], 1.0f / kLoScale, aS[t][c]);
      vI[c] = fmaf(aI[t][2 + c], 1.0f / kLoScale, aI[t][c]);
    }
    const float pre0 = vS[0] - vI[0], pre1 = vS[1] - vI[1];
    const float s_re = m == 0 ? sc[0][t][0] : sc[1][t][0], s_im = m == 0 ? sc[0][t][1] : sc[1][t][1];
    if (m == 0) {
      yr = fmaf(s_re, pre0, yr);
      yr = fmaf(-s_im, vI[1], yr);
      yi = fmaf(s_re, pre1, yi);
      yi = fmaf(s_im, vI[0], yi);
    } else {
      yr = fmaf(s_re, pre0, yr);
      yr = fmaf(s_im, vI[1], yr);
      yi = fmaf(-s_re, pre1, yi);
      yi = fmaf(s_im, vI[0], yi);
    }
  }
  return make_float2(yr, yi);
}

// y of token slot g (lane group) of a one-band tile: (yr, yi) times the token factor.
__device__ inline void store_outputs_f4(const DecLayer& L, const DecHeader& h, int row, bool row_ok, int lane,
                                        int tile, float yr, float yi, const float (&xf)[4]) {
  const int g = lane >> 4;
  const int b = 4 * tile + g;
  if (!row_ok || b >= h.B) return;
  const float f = pick_factor<4>(xf, g);
  buf_store8(L.y, (uint32_t)h.B * L.N * 8, (uint32_t)((b * L.N + row) * 8), make_float2(__fmul_rn(yr, f), __fmul_rn(yi, f)));
}

// ------------------------------------------------ per-group axis scales ---
// With per-group scales (a pair (s_re, s_im) per stage, row and group of
// 256 gsteps consecutive codes; scales [T][N][groups][2]) the MFMAs of a
// step start from zero, and the step's products, digits joined, are folded
// into float32 sums with the scales of the step's group:
//     Are += s_re (S - I),   Aim += s_im I        (per plane and component),
// so the epilogue needs no scales.  Every step's scales of both matrices
// arrive in the ring slot with the step's codes: per matrix ceil(T/2)
// direct-to-LDS dword loads, lane l of load i carrying component l % 2 of
// row (l % 32) / 2 of stage 2 i + l / 32, so the slot holds
// [matrix][stage][16 rows][s_re, s_im] with 256 bytes per load.

template <int T>
struct GroupCursor {
  const float* base[2];  // U, W scale arrays of the current layer
  uint32_t bytes;        // bytes of each array
  uint32_t tstride;      // bytes from stage t to stage t + 2
  uint32_t off;          // this lane's offset for the current step's group
  int gsteps, gpos, ngroups, N;
  bool ok;               // this lane's row and stage exist
};

template <int T>
__device__ inline void group_enter_layer(GroupCursor<T>& c, const DecLayer& L) {
  c.base[0] = L.scales[0];
  c.base[1] = L.scales[1];
  c.gsteps = L.gsteps;
  c.N = L.N;
  c.ngroups = (L.nk4 + L.gsteps - 1) / L.gsteps;
  c.bytes = (uint32_t)T * (uint32_t)L.N * (uint32_t)c.ngroups * 8u;
  c.tstride = 2u * (uint32_t)L.N * (uint32_t)c.ngroups * 8u;
}

// Position the cursor at step k4 of row block rb.
template <int T>
__device__ inline void group_item(GroupCursor<T>& c, int rb, int k4, int lane) {
  const int gi = k4 / c.gsteps;
  c.gpos = k4 - gi * c.gsteps;
  const int row = rb * 16 + ((lane & 31) >> 1);
  const int t = lane >> 5;
  c.ok = row < c.N && t < T;
  c.off = ((uint32_t)(t * c.N + row) * (uint32_t)c.ngroups + (uint32_t)gi) * 8u + 4u * (uint32_t)(lane & 1);
}

template <int T>
__device__ inline void group_step(GroupCursor<T>& c) {
  if (++c.gpos == c.gsteps) {
    c.gpos = 0;
    c.off += 8u;
  }
}

constexpr int group_loads(int T) { return (T + 1) / 2; }  // direct-to-LDS loads per matrix and step
constexpr int group_slot_bytes(int T) { return 2 * group_loads(T) * 256; }

// Issue the step's scale loads into the slot's scale area (a dead cursor
// issues them out of range, so every step issues the same number of loads).
template <int T>
__device__ inline void group_issue(const GroupCursor<T>& c, bool live, int lane, uint8_t* gslot) {
  constexpr int NI = group_loads(T);
  const int bytes = __builtin_amdgcn_readfirstlane((int)c.bytes);
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    const auto r = make_rsrc(uniform_ptr(c.base[m]), (uint32_t)bytes);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const bool v = live && c.ok && 2 * i + (lane >> 5) < T;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(gslot + (m * NI + i) * 256), 4,
                                               v ? c.off + (uint32_t)i * c.tstride : kOob, 0, 0, 0);
    }
  }
}

// Scales (s_re, s_im) of plane p = m T + t for weight row li from a slot:
// 2T LDS reads and their wait as one asm block, so that the compiler adds no
// wait of its own for the loads still in flight into the ring's other slots
// (the caller's vmcnt wait has already covered this slot).
template <int T>
__device__ inline void group_read(const uint8_t* gslot, int li, float (&gs)[2 * T][2]) {
  constexpr int NI = group_loads(T);
  const uint32_t a = lds_addr(gslot) + (uint32_t)li * 8u;
  v2f r[2 * T];
  // plane p = m T + t sits at (m NI + t / 2) * 256 + (t % 2) * 128
#define F4_GOFF(m, t) (((m) * NI + (t) / 2) * 256 + ((t) % 2) * 128)
  if constexpr (T == 1) {
    __asm__ volatile("ds_read_b64 %0, %2 offset:%3\n\tds_read_b64 %1, %2 offset:%4\n\ts_waitcnt lgkmcnt(0)"
                     : "=&v"(r[0]), "=&v"(r[1])
                     : "v"(a), "i"(F4_GOFF(0, 0)), "i"(F4_GOFF(1, 0))
                     : "memory");
  } else if constexpr (T == 2) {
    __asm__ volatile(
        "ds_read_b64 %0, %4 offset:%5\n\tds_read_b64 %1, %4 offset:%6\n\t"
        "ds_read_b64 %2, %4 offset:%7\n\tds_read_b64 %3, %4 offset:%8\n\ts_waitcnt lgkmcnt(0)"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3])
        : "v"(a), "i"(F4_GOFF(0, 0)), "i"(F4_GOFF(0, 1)), "i"(F4_GOFF(1, 0)), "i"(F4_GOFF(1, 1))
        : "memory");
  } else if constexpr (T == 3) {
    __asm__ volatile(
        "ds_read_b64 %0, %6 offset:%7\n\tds_read_b64 %1, %6 offset:%8\n\tds_read_b64 %2, %6 offset:%9\n\t"
        "ds_read_b64 %3, %6 offset:%10\n\tds_read_b64 %4, %6 offset:%11\n\tds_read_b64 %5, %6 offset:%12\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5])
        : "v"(a), "i"(F4_GOFF(0, 0)), "i"(F4_GOFF(0, 1)), "i"(F4_GOFF(0, 2)), "i"(F4_GOFF(1, 0)),
          "i"(F4_GOFF(1, 1)), "i"(F4_GOFF(1, 2))
        : "memory");
  } else {
    static_assert(T == 4, "1 <= T <= 4");
    __asm__ volatile(
        "ds_read_b64 %0, %8 offset:%9\n\tds_read_b64 %1, %8 offset:%10\n\tds_read_b64 %2, %8 offset:%11\n\t"
        "ds_read_b64 %3, %8 offset:%12\n\tds_read_b64 %4, %8 offset:%13\n\tds_read_b64 %5, %8 offset:%14\n\t"
        "ds_read_b64 %6, %8 offset:%15\n\tds_read_b64 %7, %8 offset:%16\n\ts_waitcnt lgkmcnt(0)"
        : "=&v"(r[0]), "=&v"(r[1]), "=&v"(r[2]), "=&v"(r[3]), "=&v"(r[4]), "=&v"(r[5]), "=&v"(r[6]), "=&v"(r[7])
        : "v"(a), "i"(F4_GOFF(0, 0)), "i"(F4_GOFF(0, 1)), "i"(F4_GOFF(0, 2)), "i"(F4_GOFF(0, 3)),
          "i"(F4_GOFF(1, 0)), "i"(F4_GOFF(1, 1)), "i"(F4_GOFF(1, 2)), "i"(F4_GOFF(1, 3))
        : "memory");
  }
#undef F4_GOFF
#pragma unroll
  for (int p = 0; p < 2 * T; ++p) {
    gs[p][0] = r[p][0];
    gs[p][1] = r[p][1];
  }
}

// Fold one step's products into the scaled sums (see above).
template <int P>
__device__ inline void fold_group(const v4f (&aS)[P], const v4f (&aI)[P], const float (&gs)[P][2],
                                  float (&Are)[P][2], float (&Aim)[P][2]) {
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const float vS = fmaf(aS[p][2 + c], 1.0f / kLoScale, aS[p][c]);
      const float vI = fmaf(aI[p][2 + c], 1.0f / kLoScale, aI[p][c]);
      Are[p][c] = fmaf(gs[p][0], vS - vI, Are[p][c]);
      Aim[p][c] = fmaf(gs[p][1], vI, Aim[p][c]);
    }
}

// Epilogue of a work item with per-group scales: the lane's scaled sums,
// second band passed down from the odd lane group (times 2^-8), then
// Eq. (ifairy-dequant)'s combination with the scales already applied, U
// with x and W with conj(x), stages in order, times the token factor.
template <int T, int BANDS>
__device__ inline void write_outputs_f4_gs(const DecLayer& L, const DecHeader& h, int kc, int row, bool row_ok,
                                           int lane, int tile, const float (&Are)[2 * T][2],
                                           const float (&Aim)[2 * T][2], const float (&xf)[4 / BANDS]) {
  constexpr int P = 2 * T;
  const int g = lane >> 4;
  float vr[P][2], vi[P][2];
#pragma unroll
  for (int p = 0; p < P; ++p)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      vr[p][c] = Are[p][c];
      vi[p][c] = Aim[p][c];
      if constexpr (BANDS == 2) {
        const float hr = __shfl_down(Are[p][c], 16), hi = __shfl_down(Aim[p][c], 16);
        vr[p][c] = fmaf(hr, 1.0f / kBand2Scale, Are[p][c]);
        vi[p][c] = fmaf(hi, 1.0f / kBand2Scale, Aim[p][c]);
      }
    }
  const int tt = BANDS == 2 ? g >> 1 : g;
  const int b = (4 / BANDS) * tile + tt;
  if ((BANDS == 2 && (g & 1)) || !row_ok || b >= h.B) return;
  float yr = 0.0f, yi = 0.0f;
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int u = t, w = T + t;
    yr = __fadd_rn(yr, vr[u][0]);
    yr = __fsub_rn(yr, vi[u][1]);
    yr = __fadd_rn(yr, vr[w][0]);
    yr = __fadd_rn(yr, vi[w][1]);
    yi = __fadd_rn(yi, vr[u][1]);
    yi = __fadd_rn(yi, vi[u][0]);
    yi = __fsub_rn(yi, vr[w][1]);
    yi = __fadd_rn(yi, vi[w][0]);
  }
  const float f = pick_factor<4 / BANDS>(xf, tt);
  const float2 v = make_float2(__fmul_rn(yr, f), __fmul_rn(yi, f));
  if (L.nkc == 1)
    buf_store8(L.y, (uint32_t)h.B * L.N * 8, (uint32_t)((b * L.N + row) * 8), v);
  else
    buf_store8(L.part, (uint32_t)L.nkc * h.B * L.N * 8, (uint32_t)(((kc * h.B + b) * L.N + row) * 8), v);
}

constexpr int f4_ring_slots(int T) { return ring_slots(T); }


template <int T, int XW>
using F4Cfg = StreamCfg<T, XW, f4_ring_slots(T), block_waves(T)>;

// The streaming configuration with the per-group scale area in every slot.
template <int T, int XW, bool GS>
struct F4Ring {
  using Base = F4Cfg<T, XW>;
  static constexpr int P = Base::P, NS = Base::NS;
  static constexpr int XSLOT = Base::XSLOT;                    // activation operand bytes
  static constexpr int SLOT = XSLOT + (GS ? group_slot_bytes(T) : 0);
  static constexpr int WAVES = stream_waves(NS, SLOT, block_waves(T), 1);  // fewer when the ring would not fit
  static constexpr int LOADS = Base::LOADS + (GS ? 2 * group_loads(T) : 0);
  static constexpr int WAIT = (NS - 1) * LOADS;
  static constexpr int WAITCNT = (WAIT & 0xF) | (0x7 << 4) | (0xF << 8) | (((WAIT >> 4) & 3) << 14);
  static_assert(WAIT < 64, "vmcnt holds at most 63");
};

// NT activation tiles (two tokens each); a ring slot holds XW KiB per tile.
// GS: per-group scales (every layer of the call).
template <int T, int XW, int NT, bool GS, int BANDS>
__global__ __launch_bounds__((64 * F4Ring<T, NT * XW, GS>::WAVES)) void dec_stream_f4_kernel(
    DecHeader h, DecLayer inl, const DecLayer* __restrict__ tab) {
#if defined(__HIP_DEVICE_COMPILE__)  // LDS-DMA and buffer-descriptor code: device pass only
  using C = F4Ring<T, NT * XW, GS>;
  constexpr int P = C::P, NS = C::NS, XSLOT = C::XSLOT, SLOT = C::SLOT;
  constexpr int WAVES = C::WAVES;
  static_assert(NS <= 4, "the item queue holds the items of up to NS - 1 steps ahead");
  __shared__ __attribute__((aligned(16))) uint8_t ring[WAVES][NS][SLOT];
  __shared__ __attribute__((aligned(16))) uint8_t zero16[16];
  __shared__ uint32_t claim_ctr;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, li = lane & 15;
  const int wave = uniform(threadIdx.x >> 6);
  if (threadIdx.x < 4) reinterpret_cast<uint32_t*>(zero16)[threadIdx.x] = 0u;
  if (threadIdx.x == 0) claim_ctr = (uint32_t)WAVES;  // wave w starts with item b0 + w
  __syncthreads();
  // the block's items: those starting in an equal share of the call's steps
  // (the table lists layers by decreasing item length, so a block claims its
  // longest items first and its range ends with short ones)
  // (both searches of the table advance a level per round trip, and both
  // layers are loaded together: the prologue is a chain of memory latencies)
  int64_t b0, b1;
  int la = 0;  // layer holding the block's first step
  DecLayer La = inl;
  {
    const int64_t s0 = (int64_t)blockIdx.x * h.total_steps / gridDim.x;
    const int64_t s1 = ((int64_t)blockIdx.x + 1) * h.total_steps / gridDim.x;
    if (tab) {
      const int64_t s1c = s1 < h.total_steps ? s1 : s0;
      int lo0 = 0, hi0 = h.n_layers - 1, lo1 = 0, hi1 = h.n_layers - 1;
      while (lo0 < hi0 || lo1 < hi1) {
        const int m0 = (lo0 + hi0 + 1) >> 1, m1 = (lo1 + hi1 + 1) >> 1;
        const int64_t v0 = tab[m0].step0, v1 = tab[m1].step0;
        const int64_t u0 = uniform64(v0), u1 = uniform64(v1);
        if (lo0 < hi0) {
          if (u0 <= s0) lo0 = m0;
          else hi0 = m0 - 1;
        }
        if (lo1 < hi1) {
          if (u1 <= s1c) lo1 = m1;
          else hi1 = m1 - 1;
        }
      }
      la = lo0;
      La = load_layer(tab + lo0);
      const DecLayer Lb = load_layer(tab + lo1);
      b0 = item_at_step(La, s0, h);
      b1 = item_at_step(Lb, s1, h);
    } else {
      b0 = item_at_step(inl, s0, h);
      b1 = item_at_step(inl, s1, h);
    }
  }
  b0 = uniform64(b0);
  const int nb = uniform((int)(uniform64(b1) - b0));
  if (wave >= nb) return;
  const int64_t i0 = b0 + wave;
  const uint32_t ctr_addr = lds_addr(&claim_ctr);

  // operand column li of tile t belongs to token TPT t + li / (4 BANDS)
  constexpr int TPT = 4 / BANDS;
  bool xvalid[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) xvalid[t] = TPT * t + li / (4 * BANDS) < h.B;

  LoadCursor<T> lc;
  OutCursor oc;
  GroupCursor<T> gc;
  ItemQueue iq;
  iq.n = 0;
  {
    // the wave's first item is mostly in the layer already loaded
    int lidx = la;
    DecLayer L0 = La;
    if (tab && (i0 < La.item0 || i0 >= La.item0 + (int64_t)La.nrb * La.nkc)) {
      lidx = find_layer(tab, h.n_layers, i0);
      L0 = load_layer(tab + lidx);
    }
    lc.lidx = oc.lidx = lidx;
    lc.item = oc.item = i0;
    load_enter_layer(lc, L0, h);
    out_enter_layer(oc, L0);
    if constexpr (GS) group_enter_layer(gc, L0);
    split_item(i0, lc.G, lc.rb, lc.kc);
    oc.rb = lc.rb;
    oc.kc = lc.kc;
  }
  load_item(lc, h, lane);
  if constexpr (GS) group_item(gc, lc.rb, lc.k4, lane);
  out_item(oc, li);
  // the epilogue's per-layer constants, reloaded when the output side changes layer
  float esc[2][T][2], exf[NT][TPT];
  auto load_epilogue_consts = [&]() {
    if constexpr (!GS) sload_scales<T>(uniform_ptr(oc.scales[0]), uniform_ptr(oc.scales[1]), esc);
    // the factor array is padded to 256 bytes: both floats of every tile are inside it
#pragma unroll
    for (int t = 0; t < NT; ++t) sload_run<TPT>(uniform_ptr(oc.xs) + TPT * t, exf[t]);
  };
  load_epilogue_consts();

  // next step of the load side: the next step of its item, else a claimed
  // item (queued for the output side); false once the block's items are gone
  auto load_advance = [&]() -> bool {
    if (++lc.j < lc.nsteps) {
      ++lc.k4;
      lc.voff += lc.vstep;
      lc.xoff += 256 * h.nc;
      if constexpr (GS) group_step(gc);
      return true;
    }
    const int off = claim_item(ctr_addr, nb, lane);
    if (off < 0) return false;
    const int lidx_before = lc.lidx;
    load_goto(lc, b0 + off, tab, h, lane);
    if constexpr (GS) {
      if (lc.lidx != lidx_before) group_enter_layer(gc, load_layer(tab + lc.lidx));
      group_item(gc, lc.rb, lc.k4, lane);
    }
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
  auto issue = [&](int k, v4i (&q)[P]) {
    stream_issue<XW, T, 32, NT>(lc, live, lane, q, &ring[wave][k][0]);
    if constexpr (GS) group_issue<T>(gc, live, lane, &ring[wave][k][XSLOT]);
  };
#pragma unroll
  for (int k = 0; k < NS - 1; ++k) {
    issue(k, cq[k]);
    if (live) live = load_advance();
  }

  v4f aS[NT][P], aI[NT][P];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int p = 0; p < P; ++p) aS[t][p] = aI[t][p] = v4f{0.f, 0.f, 0.f, 0.f};
  // per-group scales: the scaled sums of the current item
  float Are[NT][P][2], Aim[NT][P][2];
  if constexpr (GS) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int p = 0; p < P; ++p) Are[t][p][0] = Are[t][p][1] = Aim[t][p][0] = Aim[t][p][1] = 0.0f;
  }

  auto step = [&](auto kconst) -> bool {
    constexpr int K = decltype(kconst)::value;
    constexpr int KN = (K + NS - 1) % NS;
    issue(KN, cq[KN]);
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
          // per-group scales: every step starts from zero
          const v4f cS = (GS && kb == 0) ? v4f{0.f, 0.f, 0.f, 0.f} : aS[t][p];
          const v4f cI = (GS && kb == 0) ? v4f{0.f, 0.f, 0.f, 0.f} : aI[t][p];
          aS[t][p] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bs, cS, kFmtFp8, kFmtFp4, 0, 0, 0, 0);
          aI[t][p] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bi, cI, kFmtFp8, kFmtFp4, 0, 0, 0, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NT, 0);
      }
    }
    if constexpr (GS) {
      float gs[P][2];
      group_read<T>(&ring[wave][K][XSLOT], li, gs);
#pragma unroll
      for (int t = 0; t < NT; ++t) fold_group<P>(aS[t], aI[t], gs, Are[t], Aim[t]);
    }
    if (oc.j == oc.nsteps - 1) {
      const DecLayer Lo = out_layer(oc);
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if constexpr (GS) {
          write_outputs_f4_gs<T, BANDS>(Lo, h, oc.kc, oc.row, oc.row_ok, lane, t, Are[t], Aim[t], exf[t]);
#pragma unroll
          for (int p = 0; p < P; ++p) Are[t][p][0] = Are[t][p][1] = Aim[t][p][0] = Aim[t][p][1] = 0.0f;
        } else {
          write_outputs_f4<T, BANDS>(Lo, h, oc.kc, oc.row, oc.row_ok, lane, t, aS[t], aI[t], esc, exf[t]);
#pragma unroll
          for (int p = 0; p < P; ++p) aS[t][p] = aI[t][p] = v4f{0.f, 0.f, 0.f, 0.f};
        }
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

template <int T, int XW, int NT, bool GS, int BANDS>
void launch_stream_f4(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s) {
  auto k = dec_stream_f4_kernel<T, XW, NT, GS, BANDS>;
  constexpr int waves = F4Ring<T, NT * XW, GS>::WAVES;
  constexpr int threads = 64 * waves;
  static const int resident = resident_blocks(reinterpret_cast<const void*>(k), threads);
  const int64_t want = (h.total_items + waves - 1) / waves;
  const int64_t blocks = want < resident ? want : resident;
  hipLaunchKernelGGL(k, dim3((unsigned)blocks), dim3(threads), 0, s, h, inl, tab);
}

// XW = KiB of activation operand per 256-code step and tile (nc / 4), NT =
// activation tiles of two tokens (three or four tokens: two tiles, T <= 3).
// One tile: one token (two bands, 8 columns), two tokens (two bands) or
// three to four (one band); two tiles: five to eight tokens (one band,
// T <= 3); four tiles: nine to sixteen tokens (one band, T <= 2).
template <int T, bool GS>
void launch_stream_f4_g(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s) {
  if constexpr (T <= 2) {
    if (h.ntile >= 3) {
      launch_stream_f4<T, 4, 4, GS, 1>(h, inl, tab, s);
      return;
    }
  }
  if constexpr (T <= 3) {
    if (h.ntile >= 2) {
      if (h.bands == 2) launch_stream_f4<T, 4, 2, GS, 2>(h, inl, tab, s);
      else launch_stream_f4<T, 4, 2, GS, 1>(h, inl, tab, s);
      return;
    }
  }
  if (h.nc <= 8) launch_stream_f4<T, 2, 1, GS, 2>(h, inl, tab, s);
  else if (h.bands == 2) launch_stream_f4<T, 4, 1, GS, 2>(h, inl, tab, s);
  else launch_stream_f4<T, 4, 1, GS, 1>(h, inl, tab, s);
}

template <int T, int NT, int NC, int BANDS, bool GS>
void launch_coop_f4(const DecHeader& h, const DecLayer* tab, hipStream_t s);  // the block-cooperative kernel below

// The cooperative kernel for one or two tiles (per-group scales or not).
template <int T, bool GS>
void launch_coop_f4_small(const DecHeader& h, const DecLayer* tab, hipStream_t s) {
  if (h.ntile == 2) {
    if (h.bands == 2) launch_coop_f4<T, 2, 16, 2, GS>(h, tab, s);
    else launch_coop_f4<T, 2, 16, 1, GS>(h, tab, s);
  } else if (h.nc <= 8) {
    launch_coop_f4<T, 1, 8, 2, GS>(h, tab, s);
  } else if (h.bands == 2) {
    launch_coop_f4<T, 1, 16, 2, GS>(h, tab, s);
  } else {
    launch_coop_f4<T, 1, 16, 1, GS>(h, tab, s);
  }
}
constexpr bool kCoopSmallB = true;  // one tile (1-4 tokens) on the cooperative kernel too

template <int T>
void launch_stream_f4_t(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s) {
  if (h.grouped) {
    if constexpr (T <= 2) {
      if (tab && h.coop && h.ntile <= 2) {
        launch_coop_f4_small<T, true>(h, tab, s);
        return;
      }
    }
    launch_stream_f4_g<T, true>(h, inl, tab, s);
    return;
  }
  if constexpr (T <= 2) {
    if (tab && h.coop && h.ntile >= 3) {
      launch_coop_f4<T, 4, 16, 1, false>(h, tab, s);
      return;
    }
    if (tab && h.coop && (h.ntile == 2 || kCoopSmallB)) {
      launch_coop_f4_small<T, false>(h, tab, s);
      return;
    }
  }
  launch_stream_f4_g<T, false>(h, inl, tab, s);
}

// ------------------------------------------- block-cooperative kernel ---
// A per-wave ring holds a copy of each step's activation operand per wave;
// with five or more tokens that operand (NT tiles of 4 KiB) outweighs the
// step's codes (2T KiB) and leaves room for few waves per CU, and even with
// one token every wave fetches it from L2 again.  Here the waves of a block
// decode consecutive row blocks of one layer (a group) together, stepping
// through K in lockstep (with four tiles two waves share a row block, two
// tiles each).  One ring of kCoopSlots slots in LDS holds each step's
// activation operand once for the whole block (each wave loads its share),
// the codes go to each wave's own registers as in the streaming kernel, and
// one barrier per step both publishes the slot about to be read and retires
// the slot read the step before (the one the step's new loads overwrite).
// Blocks take the groups that start in an equal share of the call's group
// steps; the table lists layers by decreasing length.  Used when every layer
// is one full-K item per row block (no partials).
//
// Blocks that share a CU do not progress at the same rate (the waves of the
// block dispatched first are served first), so with static shares alone the
// first blocks finish early and the last ones leave the chip half idle.  The
// last groups (the shortest) are therefore claimed at run time: when a
// block's load cursor starts its last known group, lane 0 of wave 0 takes a
// ticket from a global counter; the ticket returns with that step's loads,
// is read kCoopSlots - 1 steps later after the step's wait, translated to a
// (group, layer) pair and posted in LDS, where every wave reads it after the
// next barrier.  That needs groups longer than kCoopSlots steps (the host
// enables claims only then).  A group's outputs do not depend on which block
// decodes it.

// Global index of the first group (of rbg row blocks) whose first step is at
// or after group step s.
__device__ inline int64_t coop_group_at_step(const DecLayer* tab, int n, int64_t s, int64_t total, int rbg) {
  if (s >= total) {
    const int64_t g0 = uniform64(tab[n - 1].sitem0);
    return g0 + (uniform(tab[n - 1].nrb) + rbg - 1) / rbg;
  }
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (uniform64(tab[mid].sstep0) <= s) lo = mid;
    else hi = mid - 1;
  }
  const int nk4 = uniform(tab[lo].nk4);
  return uniform64(tab[lo].sitem0) + (s - uniform64(tab[lo].sstep0) + nk4 - 1) / nk4;
}

// Layer holding global group q: the last layer whose sitem0 <= q.
__device__ inline int coop_layer_of_group(const DecLayer* tab, int n, int64_t q) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (uniform64(tab[mid].sitem0) <= q) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Wave-uniform position in the block's sequence of (group, step).
struct CoopCursor {
  int64_t q, qend;  // global group, one past the block's last
  const uint8_t* codes[2];
  const int8_t* xf;
  int lidx;
  int g, k4;        // group within the layer, step within the group
  int ngroups, nk4, nrb, N, K, rbg;
  bool live;
};

__device__ inline void coop_enter_layer(CoopCursor& c, const DecLayer& L) {
  c.codes[0] = L.codes[0];
  c.codes[1] = L.codes[1];
  c.xf = L.xf;
  c.nk4 = L.nk4;
  c.nrb = L.nrb;
  c.N = L.N;
  c.K = L.K;
  c.ngroups = (L.nrb + c.rbg - 1) / c.rbg;
}

// A claimed group as posted in LDS by wave 0: global group index (past the
// last group: nothing left) and its layer.
struct __attribute__((aligned(16))) CoopPost {
  int64_t q;
  int32_t lidx, pad_;
};

// Next step; enters the next group / layer (reading its descriptor).  Past
// the block's known groups: the claimed group posted in LDS, if claims run.
__device__ inline void coop_advance(CoopCursor& c, const DecLayer* tab, const DecHeader& h, const CoopPost* post) {
  if (++c.k4 < c.nk4) return;
  c.k4 = 0;
  ++c.q;
  if (c.q >= c.qend) {
    if (h.coop_dyn0 >= h.coop_groups) {
      c.live = false;
      return;
    }
    int64_t q;
    int l;
    asm volatile(
        "ds_read_b64 %0, %2\n"
        "ds_read_b32 %1, %2 offset:8\n"
        "s_waitcnt lgkmcnt(0)"
        : "=v"(q), "=v"(l)
        : "v"(lds_addr(post))
        : "memory");
    q = uniform64(q);
    if (q >= h.coop_groups) {
      c.live = false;
      return;
    }
    c.q = q;
    c.qend = q + 1;
    c.lidx = uniform(l);
    const DecLayer L = load_layer(tab + c.lidx);
    coop_enter_layer(c, L);
    c.g = (int)(q - L.sitem0);
    return;
  }
  if (++c.g == c.ngroups) {
    c.g = 0;
    ++c.lidx;
    coop_enter_layer(c, load_layer(tab + c.lidx));
  }
}

// A step's activation reads for one wave: both 128-code halves (kb) of TS
// tiles, two 16-byte reads each, issued together; with one tile the asm waits
// for the first half's reads, with two the first half's tiles are waited for
// one at a time (coop_wait_tile, as with four tiles), and coop_wait_x waits
// for the rest, so the second half's LDS latency hides behind the first
// half's MFMAs.  Registers that a later wait covers pass through it as
// in/out operands, which keeps every use of them after that wait.
template <int TS>
__device__ inline void coop_read_x(const uint32_t (&a)[2][TS][2], v4i (&x)[2][TS][2]) {
  static_assert(TS == 1 || TS == 2, "one or two tiles per wave");
  if constexpr (TS == 1) {
    __asm__ volatile(
        "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\tds_read_b128 %3, %7\n\t"
        "s_waitcnt lgkmcnt(2)"
        : "=&v"(x[0][0][0]), "=&v"(x[0][0][1]), "=&v"(x[1][0][0]), "=&v"(x[1][0][1])
        : "v"(a[0][0][0]), "v"(a[0][0][1]), "v"(a[1][0][0]), "v"(a[1][0][1])
        : "memory");
  } else {
    __asm__ volatile(
        "ds_read_b128 %0, %8\n\tds_read_b128 %1, %9\n\tds_read_b128 %2, %10\n\tds_read_b128 %3, %11\n\t"
        "ds_read_b128 %4, %12\n\tds_read_b128 %5, %13\n\tds_read_b128 %6, %14\n\tds_read_b128 %7, %15"
        : "=&v"(x[0][0][0]), "=&v"(x[0][0][1]), "=&v"(x[0][1][0]), "=&v"(x[0][1][1]), "=&v"(x[1][0][0]),
          "=&v"(x[1][0][1]), "=&v"(x[1][1][0]), "=&v"(x[1][1][1])
        : "v"(a[0][0][0]), "v"(a[0][0][1]), "v"(a[0][1][0]), "v"(a[0][1][1]), "v"(a[1][0][0]), "v"(a[1][0][1]),
          "v"(a[1][1][0]), "v"(a[1][1][1])
        : "memory");
  }
}

// Four tiles: one 128-code half's eight reads (the halves one after the
// other, so that only one half's operands are live), issued without a wait;
// coop_wait_tile<6 - 2t> then waits for tile t alone (LDS reads complete in order),
// so a tile's MFMAs start while the later tiles' reads are still served.
// After a step's barrier every wave of the block reads the whole operand at
// once, which keeps the LDS busy for several hundred cycles.  Tile t's
// registers pass through its wait as in/out operands, which keeps every use
// of them after that wait.
__device__ inline void coop_read_x4(const uint32_t (&a)[4][2], v4i (&x)[4][2]) {
  __asm__ volatile(
      "ds_read_b128 %0, %8\n\tds_read_b128 %1, %9\n\tds_read_b128 %2, %10\n\tds_read_b128 %3, %11\n\t"
      "ds_read_b128 %4, %12\n\tds_read_b128 %5, %13\n\tds_read_b128 %6, %14\n\tds_read_b128 %7, %15"
      : "=&v"(x[0][0]), "=&v"(x[0][1]), "=&v"(x[1][0]), "=&v"(x[1][1]), "=&v"(x[2][0]), "=&v"(x[2][1]),
        "=&v"(x[3][0]), "=&v"(x[3][1])
      : "v"(a[0][0]), "v"(a[0][1]), "v"(a[1][0]), "v"(a[1][1]), "v"(a[2][0]), "v"(a[2][1]), "v"(a[3][0]),
        "v"(a[3][1])
      : "memory");
}


// Wait until at most N of the LDS reads issued before are outstanding (one
// tile's two registers covered).
template <int N>
__device__ inline void coop_wait_tile(v4i (&x)[2]) {
  __asm__ volatile("s_waitcnt lgkmcnt(%2)" : "+v"(x[0]), "+v"(x[1]) : "i"(N) : "memory");
}

template <int TS>
__device__ inline void coop_wait_x(v4i (&x)[2][TS][2]) {
  if constexpr (TS == 1) {
    __asm__ volatile("s_waitcnt lgkmcnt(0)" : "+v"(x[1][0][0]), "+v"(x[1][0][1]) : : "memory");
  } else {
    __asm__ volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(x[1][0][0]), "+v"(x[1][0][1]), "+v"(x[1][1][0]), "+v"(x[1][1][1])
                     :
                     : "memory");
  }
}

// Every wave multiplies all NT activation tiles.  PS waves share a row
// block, each taking P / PS of its code planes: with four tiles (PS = 2) one
// wave takes the U planes and one the W planes, so a wave's accumulators
// stay at 64 registers and each code byte is still loaded and expanded once;
// the two halves of y meet in LDS at the end of a group.
// NC columns per tile (8: one two-band token; 16), BANDS digit bands per token.
// GS: per-group scales (every layer of the call; one or two tiles): each
// wave's row block has its step's scales loaded into the ring slot with the
// step's operands, every step's products start from zero and are folded into
// scaled float32 sums (as in the streaming kernel).
template <int T, int NT, int PS, int NC, int BANDS, bool GS>
__global__ __launch_bounds__(64 * coop_waves(NT), coop_waves(NT) == 8 ? 1 : 2) void dec_coop_f4_kernel(DecHeader h,
                                                                      const DecLayer* __restrict__ tab) {
#if defined(__HIP_DEVICE_COMPILE__)  // LDS-DMA and buffer-descriptor code: device pass only
  constexpr int P = 2 * T;
  constexpr int TS = NT;                // tiles per wave
  constexpr int PW = P / PS;            // code planes per wave
  constexpr int W = coop_waves(NT);
  constexpr int RBG = W / PS;           // row blocks per group
  static_assert(P % PS == 0 && W % PS == 0, "planes split evenly over the waves of a row block");
  static_assert(PS == 1 || (PS == 2 && BANDS == 1), "split planes: one-band tiles only");
  static_assert(TS == 1 || TS == 2 || TS == 4, "one, two or four tiles");
  static_assert(!GS || PS == 1, "per-group scales: one wave per row block");
  constexpr int GSB = GS ? group_slot_bytes(T) : 16;  // a wave's scale bytes per step
  constexpr int NS = kCoopSlots;
  constexpr int XT = NC * 256;          // a tile's operand per step: NC columns x 256 codes
  constexpr int XS = NT * XT;           // a step's activation operand
  constexpr int NDMA = XS / 1024;       // its 1-KiB loads
  constexpr int DMA = (NDMA + W - 1) / W;  // per wave (waves past the last load issue an empty one)
  constexpr int TPT = 4 / BANDS;        // tokens per 16 columns
  constexpr int CPT = 4 * BANDS;        // columns per token
  constexpr int LOADS = PW + DMA + (GS ? 2 * group_loads(T) : 0);  // vector memory ops per wave and step
  constexpr int WAIT = (NS - 2) * LOADS;  // when step j is read, steps j+1 .. j+NS-2 may still load
  constexpr int WAITCNT = (WAIT & 0xF) | (0x7 << 4) | (0xF << 8) | (((WAIT >> 4) & 3) << 14);
  static_assert(WAIT < 64, "vmcnt holds at most 63");
  __shared__ __attribute__((aligned(16))) uint8_t ring[NS][XS];
  __shared__ __attribute__((aligned(16))) uint8_t zero16[16];
  // target of the empty loads of waves past the step's last activation load
  // (an out-of-range load still writes its zeros to LDS)
  __shared__ __attribute__((aligned(16))) uint8_t spare[NDMA % W ? 1024 : 16];
  __shared__ CoopPost post;
  // per-group scales: [slot][wave] scale area of each step
  __shared__ __attribute__((aligned(16))) uint8_t gring[GS ? NS : 1][GS ? W : 1][GSB];
  // split planes: the W waves' partial outputs, [row block][tile][lane] (re, im)
  __shared__ __attribute__((aligned(16))) float2 xch[PS == 2 ? RBG * TS * 64 : 1];
  const int lane = threadIdx.x & 63;
  const int g4 = lane >> 4, li = lane & 15;
  const int wave = uniform(threadIdx.x >> 6);
  if (threadIdx.x < 4) reinterpret_cast<uint32_t*>(zero16)[threadIdx.x] = 0u;
  __syncthreads();

  // the block's groups: those starting in an equal share of the statically
  // split group steps, then (with claims) groups claimed at run time
  const bool dyn = h.coop_dyn0 < h.coop_groups;
  const int64_t s0 = (int64_t)blockIdx.x * h.coop_dyn_steps / gridDim.x;
  const int64_t s1 = ((int64_t)blockIdx.x + 1) * h.coop_dyn_steps / gridDim.x;
  int64_t q0 = uniform64(coop_group_at_step(tab, h.n_layers, s0, h.total_ssteps, RBG));
  int64_t q1 = uniform64(coop_group_at_step(tab, h.n_layers, s1, h.total_ssteps, RBG));
  if (q0 >= q1) {
    if (!dyn) return;  // the whole block leaves before its first barrier
    // no static share: claim the first group now
    if (threadIdx.x == 0) post.q = h.coop_dyn0 + (int64_t)atomicAdd(h.coop_ctr, 1u);
    __syncthreads();
    q0 = uniform64(post.q);
    if (q0 >= h.coop_groups) return;  // nothing left: the whole block leaves
    q1 = q0 + 1;
  }
  const int wrb = wave / PS;              // this wave's row block within a group
  const int pw0 = (wave % PS) * PW;       // and its first code plane

  CoopCursor lc;
  {
    lc.rbg = RBG;
    lc.q = q0;
    lc.qend = q1;
    lc.lidx = coop_layer_of_group(tab, h.n_layers, q0);
    const DecLayer L0 = load_layer(tab + lc.lidx);
    coop_enter_layer(lc, L0);
    lc.g = (int)(q0 - L0.sitem0);
    lc.k4 = 0;
    lc.live = true;
  }
  CoopCursor oc = lc;

  // the claim in flight (wave 0; at most one, since claims are a group
  // apart): the ring slot whose loads carried it, and a ticket register per
  // slot (so that the compiler sees each ticket written a ring round before
  // it is read or overwritten, and adds no wait of its own)
  uint32_t cret[NS];
  int cslot = -1;

  // issue the loads of the load cursor's step into slot k: this wave's codes
  // (registers cq) and its share of the activation operand (LDS).  At the
  // first step of the block's last known group wave 0 also claims the next
  // group; the claim goes out before the slot's loads, so the wait for them
  // covers it.
  GroupCursor<T> gc;
  int glidx = -1;  // the layer gc was entered for
  auto issue = [&](int k, v4i (&cq)[PW]) {
    if constexpr (GS) {
      if (lc.live && lc.k4 == 0) {
        if (lc.lidx != glidx) {
          group_enter_layer(gc, load_layer(tab + lc.lidx));
          glidx = lc.lidx;
        }
        group_item(gc, lc.g * RBG + wrb, 0, lane);
      }
      group_issue<T>(gc, lc.live, lane, &gring[k][wave][0]);
      group_step(gc);
    }
    if (dyn && wave == 0 && lc.live && lc.k4 == 0 && lc.q + 1 >= lc.qend) {
      // one lane's atomic without a divergent branch: the other lanes' offsets
      // are out of range, so their adds are dropped
      cret[k] = (uint32_t)__builtin_amdgcn_raw_ptr_buffer_atomic_add_i32(1, make_rsrc(h.coop_ctr, 4u),
                                                                         lane == 0 ? 0u : kOob, 0, 0);
      cslot = k;
    }
    const int rb = lc.g * RBG + wrb;
    const bool ok = lc.live && rb < lc.nrb && rb * 16 + li < lc.N && lc.k4 * 256 + 32 * g4 < lc.K;
    const uint32_t pb = (uint32_t)(T * lc.nrb * lc.nk4 * 1024) - (uint32_t)(T - 1) * 1024u;
    const uint32_t off = ok ? (uint32_t)((rb * lc.nk4 + lc.k4) * T) * 1024u + (uint32_t)lane * 16u : kOob;
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int p = pw0 + j;
      // a select, not an index: a cursor indexed by a run-time value would live in scratch memory
      const uint8_t* cm = p < T ? lc.codes[0] : lc.codes[1];
      cq[j] = __builtin_amdgcn_raw_buffer_load_b128(make_rsrc(uniform_ptr(cm + (p % T) * 1024), pb), off, 0,
                                                    kNonTemporal);
    }
    const uint32_t xtile = (uint32_t)(lc.nk4 * XT);
    const auto xr = make_rsrc(uniform_ptr(lc.xf), (uint32_t)(h.ntile * xtile));
#pragma unroll
    for (int i = 0; i < DMA; ++i) {
      const int d0 = wave * DMA + i;
      const bool real = d0 < NDMA;
      const int d = real ? d0 : 0, t = d / (XT / 1024), c = d % (XT / 1024);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          xr, (lds_ptr_t)(real ? &ring[k][t * XT + c * 1024] : &spare[0]), 16,
          lc.live && real ? (uint32_t)t * xtile + (uint32_t)(lc.k4 * XT + c * 1024 + lane * 16) : kOob, 0, 0, 0);
    }
  };

  // the epilogue's per-layer constants of the output cursor's layer
  float esc[2][T][2], exf[TS][TPT];
  DecLayer Lo;
  auto load_out_layer = [&]() {
    Lo = load_layer(tab + oc.lidx);
    sload_scales<T>(uniform_ptr(Lo.scales[0]), uniform_ptr(Lo.scales[1]), esc);
#pragma unroll
    for (int t = 0; t < TS; ++t) sload_run<TPT>(uniform_ptr(Lo.xs) + TPT * t, exf[t]);
  };
  load_out_layer();

  bool xvalid[TS];
#pragma unroll
  for (int t = 0; t < TS; ++t) xvalid[t] = li < NC && TPT * t + li / CPT < h.B;

  v4i cq[NS][PW];
#pragma unroll
  for (int k = 0; k < NS - 1; ++k) {
    issue(k, cq[k]);
    if (lc.live) coop_advance(lc, tab, h, &post);
  }
  v4f aS[TS][PW], aI[TS][PW];
#pragma unroll
  for (int t = 0; t < TS; ++t)
#pragma unroll
    for (int j = 0; j < PW; ++j) aS[t][j] = aI[t][j] = v4f{0.f, 0.f, 0.f, 0.f};
  // per-group scales: the scaled sums of the current group
  float Are[TS][PW][2], Aim[TS][PW][2];
  if constexpr (GS) {
#pragma unroll
    for (int t = 0; t < TS; ++t)
#pragma unroll
      for (int j = 0; j < PW; ++j) Are[t][j][0] = Are[t][j][1] = Aim[t][j][0] = Aim[t][j][1] = 0.0f;
  }

  auto step = [&](auto kconst) -> bool {
    constexpr int K = decltype(kconst)::value;
    constexpr int KN = (K + NS - 1) % NS;  // the slot read the step before
    __builtin_amdgcn_s_waitcnt(WAITCNT);   // this wave's loads of slot K are done
    __builtin_amdgcn_s_barrier();           // every wave's loads of slot K are done; slot KN is free
    if (uniform(cslot) == K) {
      // wave 0: the claim sent with slot K's loads has returned (the wait
      // above covers it); post it for every wave (read at the load cursor's
      // next group change, which comes at least one barrier later).  The
      // ticket is read here, in order, so that no earlier read of it forces
      // a wait for every load in flight.
      cslot = -1;
      uint32_t t;
      asm volatile("v_readfirstlane_b32 %0, %1" : "=s"(t) : "v"(cret[K]));
      const int64_t q = h.coop_dyn0 + (int64_t)t;
      const int l = q < h.coop_groups ? coop_layer_of_group(tab, h.n_layers, q) : 0;
      if (lane == 0)
        asm volatile(
            "ds_write_b64 %0, %1\n"
            "ds_write_b32 %0, %2 offset:8\n"
            "s_waitcnt lgkmcnt(0)"
            :
            : "v"(lds_addr(&post)), "v"(q), "v"(l)
            : "memory");
    }
    issue(KN, cq[KN]);
    if (lc.live) coop_advance(lc, tab, h, &post);
    const v4i* cr = cq[K];
    uint32_t xa[2][TS][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int t = 0; t < TS; ++t) {
        const uint32_t a = xvalid[t] ? lds_addr(&ring[K][t * XT]) + (uint32_t)((g4 * NC + li) * 16) +
                                           kb * (uint32_t)(2 * 64 * NC)
                                     : lds_addr(zero16);
        xa[kb][t][0] = a;
        xa[kb][t][1] = a + (xvalid[t] ? (uint32_t)(64 * NC) : 0u);
      }
    // the halves' operands: both read up front (one or two tiles), else one
    // half at a time (four tiles)
    v4i xq[TS == 4 ? 1 : 2][TS][2];
    if constexpr (TS != 4) coop_read_x<TS>(xa, xq);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      if constexpr (TS == 4) {
        coop_read_x4(xa[kb], xq[0]);
      } else if (kb == 1) {
        // the first half's MFMAs stay ahead of the second half's wait
        __builtin_amdgcn_sched_barrier(0);
        coop_wait_x<TS>(xq);
      }
      v4i(&xr)[TS][2] = xq[TS == 4 ? 0 : kb];
#pragma unroll
      for (int j = 0; j < PW; ++j) {
        v8i bs, bi;
        expand_f4((uint32_t)cr[j][2 * kb], (uint32_t)cr[j][2 * kb + 1], bs, bi);
#pragma unroll
        for (int t = 0; t < TS; ++t) {
          if constexpr (TS == 4) {
            if (j == 0) {
              // the earlier tiles' MFMAs stay ahead of this tile's wait
              if (t > 0) __builtin_amdgcn_sched_barrier(0);
              if (t == 0) coop_wait_tile<6>(xr[0]);
              else if (t == 1) coop_wait_tile<4>(xr[1]);
              else if (t == 2) coop_wait_tile<2>(xr[2]);
              else coop_wait_tile<0>(xr[3]);
            }
          } else if constexpr (TS == 2) {
            // the first half's tiles (the second half's four reads were issued after them)
            if (kb == 0 && j == 0) {
              if (t > 0) __builtin_amdgcn_sched_barrier(0);
              if (t == 0) coop_wait_tile<6>(xr[0]);
              else coop_wait_tile<4>(xr[1]);
            }
          }
          const v4i x0 = xr[t][0], x1 = xr[t][1];
          const v8i a = v8i{x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
          // per-group scales: every step starts from zero
          const v4f cS = (GS && kb == 0) ? v4f{0.f, 0.f, 0.f, 0.f} : aS[t][j];
          const v4f cI = (GS && kb == 0) ? v4f{0.f, 0.f, 0.f, 0.f} : aI[t][j];
          aS[t][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bs, cS, kFmtFp8, kFmtFp4, 0, 0, 0, 0);
          aI[t][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bi, cI, kFmtFp8, kFmtFp4, 0, 0, 0, 0);
        }
        // one plane's expansion, then its MFMAs: bounds the registers the schedule keeps live
        __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * TS, 0);
      }
    }
    if constexpr (GS) {
      float gs[PW][2];
      group_read<T>(&gring[K][wave][0], li, gs);
#pragma unroll
      for (int t = 0; t < TS; ++t) fold_group<PW>(aS[t], aI[t], gs, Are[t], Aim[t]);
    }
    if (oc.k4 == oc.nk4 - 1) {
      const int rb = oc.g * RBG + wrb;
      const int row = rb * 16 + li;
      const bool row_ok = rb < oc.nrb && row < oc.N;
      if constexpr (GS) {
#pragma unroll
        for (int t = 0; t < TS; ++t) {
          write_outputs_f4_gs<T, BANDS>(Lo, h, 0, row, row_ok, lane, t, Are[t], Aim[t], exf[t]);
#pragma unroll
          for (int j = 0; j < PW; ++j) Are[t][j][0] = Are[t][j][1] = Aim[t][j][0] = Aim[t][j][1] = 0.0f;
        }
      } else if constexpr (PS == 1) {
#pragma unroll
        for (int t = 0; t < TS; ++t)
          write_outputs_f4<T, BANDS>(Lo, h, 0, row, row_ok, lane, t, aS[t], aI[t], esc, exf[t]);
      } else {
        // the W wave posts its half of y in LDS, the U wave adds it and writes y
        const int m = pw0 / T;
        float2 part[TS];
#pragma unroll
        for (int t = 0; t < TS; ++t) part[t] = partial_outputs_f4<T>(m, aS[t], aI[t], esc);
        const uint32_t xa = lds_addr(&xch[(wrb * TS) * 64 + lane]);
        if (m == 1) {
#pragma unroll
          for (int t = 0; t < TS; ++t)
            asm volatile("ds_write_b64 %0, %1 offset:%2" : : "v"(xa), "v"(part[t]), "i"(t * 512) : "memory");
          asm volatile("s_waitcnt lgkmcnt(0)" : : : "memory");
        }
        __builtin_amdgcn_s_barrier();
        if (m == 0) {
#pragma unroll
          for (int t = 0; t < TS; ++t) {
            float2 o;
            asm volatile("ds_read_b64 %0, %1 offset:%2\n\ts_waitcnt lgkmcnt(0)" : "=v"(o) : "v"(xa), "i"(t * 512)
                         : "memory");
            store_outputs_f4(Lo, h, row, row_ok, lane, t, part[t].x + o.x, part[t].y + o.y, exf[t]);
          }
        }
        // the next group's posts come after the next step's barrier, which
        // every U wave reaches only after these reads
      }
#pragma unroll
      for (int t = 0; t < TS; ++t)
#pragma unroll
        for (int j = 0; j < PW; ++j) aS[t][j] = aI[t][j] = v4f{0.f, 0.f, 0.f, 0.f};
    }
    const int lbefore = oc.lidx;
    if (dyn) {
      // the load cursor runs kCoopSlots - 1 steps ahead through the same
      // groups, each longer than that: at a group change it is in the next one
      if (++oc.k4 == oc.nk4) {
        oc = lc;
        oc.k4 = 0;
      }
    } else {
      coop_advance(oc, tab, h, &post);
    }
    if (!oc.live) return true;
    if (oc.lidx != lbefore) load_out_layer();
    return false;
  };

  static_assert(NS == 3 || NS == 4, "the ring loop below is unrolled for 3 or 4 slots");
  while (true) {
    if (step(std::integral_constant<int, 0>{})) break;
    if (step(std::integral_constant<int, 1>{})) break;
    if (step(std::integral_constant<int, 2>{})) break;
    if constexpr (NS == 4) if (step(std::integral_constant<int, 3 % NS>{})) break;
  }
  __builtin_amdgcn_s_waitcnt(0);  // no load may still be writing LDS when the wave ends
#endif
}

template <int T, int NT, int NC, int BANDS, bool GS>
void launch_coop_f4(const DecHeader& h, const DecLayer* tab, hipStream_t s) {
  auto k = dec_coop_f4_kernel<T, NT, coop_plane_split(NT), NC, BANDS, GS>;
  static const int resident = resident_blocks(reinterpret_cast<const void*>(k), 64 * coop_waves(NT));
  hipLaunchKernelGGL(k, dim3((unsigned)resident), dim3(64 * coop_waves(NT)), 0, s, h, tab);
}

}  // namespace

void launch_f4_prep(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s) {
  // up to four two-band tokens: one block per layer and token slot (its work
  // is a latency chain, not throughput)
  if (h.B <= 4 && h.bands == 2 && h.nc == (h.B == 1 ? 8 : 16) && h.ntile == (h.B + 1) / 2 && h.max_nk4 > 0) {
    const dim3 g((unsigned)h.n_layers, (unsigned)(h.B == 1 ? 1 : 2 * h.ntile)), b(kPrepF4Threads);
    const int kmax = h.max_nk4 * 256;  // entries of the longest token, padded to whole steps
    if (kmax <= 4 * kPrepF4Threads) {
      hipLaunchKernelGGL(dec_prep_f4_token_kernel<4>, g, b, 0, s, h, inl, tab);
      return;
    }
    if (kmax <= 8 * kPrepF4Threads) {
      hipLaunchKernelGGL(dec_prep_f4_token_kernel<8>, g, b, 0, s, h, inl, tab);
      return;
    }
    if (kmax <= 16 * kPrepF4Threads) {
      hipLaunchKernelGGL(dec_prep_f4_token_kernel<16>, g, b, 0, s, h, inl, tab);
      return;
    }
  }
  const int slices = (h.B == 1 || h.ntile >= kPrepF4Blocks) ? 1 : kPrepF4Blocks / h.ntile;
  hipLaunchKernelGGL(dec_prep_f4_kernel, dim3(h.ntile, h.n_layers, slices), dim3(kPrepF4Threads), 0, s, h, inl, tab);
}

void launch_f4_product(const DecHeader& h, const DecLayer& inl, const DecLayer* tab, hipStream_t s) {
  switch (h.T) {
    case 1: launch_stream_f4_t<1>(h, inl, tab, s); break;
    case 2: launch_stream_f4_t<2>(h, inl, tab, s); break;
    case 3: launch_stream_f4_t<3>(h, inl, tab, s); break;
    default: launch_stream_f4_t<4>(h, inl, tab, s); break;
  }
}

}  // namespace fairy2i
