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
#include "decode_dev.h"

namespace fairy2i {

namespace {

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


// ----------------------------------------------------------------- prep ---
constexpr int kPrepSplit = 4;

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
  if constexpr (MODE == kModeBf16) {
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
        e = 22 - ex;          // g * 2^e in [2^21, 2^22): 3 base-256 digits
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
    launch_f4_prep(h, inl, tab, s);
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
    // one or two activation tiles, codes in the fp4 tiled layout: checked by the host code
    launch_f4_product(h, inl, tab, s);
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

// fp4 path: two digit bands per value (8 columns per token, two tokens per
// tile; exact for any bf16 token) while the tokens fit the two-tile kernels
// that exist for T (up to 2 tokens, and up to 4 for T <= 3), else one band
// (4 columns per token, four tokens per tile).
int dec_f4_bands(int T, int64_t B) { return (B <= 2 || (B <= 4 && T <= 3)) ? 2 : 1; }

int dec_ntile(int mode, int64_t B, int T) {
  if (mode == kModeI8) return (int)((B + 7) / 8);
  if (mode == kModeBf16F4) return dec_f4_bands(T, B) == 2 ? (int)((B + 1) / 2) : (int)((B + 3) / 4);
  return (int)((B + 1) / 2);
}

int dec_ncols(int mode, int64_t B) {
  if (mode == kModeBf16) return B >= 2 ? 14 : 6;  // per token 6 digit columns, 8-column stride
  if (mode == kModeBf16F4) return B == 1 ? 8 : 16;  // 8 columns per two-band token, 4 per one-band token
  return B >= 8 ? 16 : (int)(2 * B);
}

DecHeader dec_header(int T, int mode, int64_t B, bool export_acc) {
  DecHeader h{};
  h.T = T;
  h.mode = mode;
  h.B = (int32_t)B;
  h.ntile = dec_ntile(mode, B, T);
  h.nc = dec_ncols(mode, B);
  h.bands = mode == kModeBf16F4 ? dec_f4_bands(T, B) : 1;
  // the fp4 path always runs its streaming kernel (one or two tiles)
  h.kernel = (!export_acc && (h.ntile == 1 || mode == kModeBf16F4)) ? kKernelStream : kKernelReg;
  return h;
}

size_t dec_layer_setup(DecLayer& l, const DecHeader& h, bool single, char* ws, int slice) {
  l.nrb = (int32_t)((l.N + 15) / 16);
  l.nk4 = (int32_t)((l.K + 255) / 256);
  if (h.kernel == kKernelReg) {
    l.kc4 = kRegKc4;
  } else if (slice == kSliceFullK && l.nk4 <= kMaxFullKSteps) {
    l.kc4 = l.nk4;  // one work item per row block
  } else {
    // slices of up to 8 steps (2048 codes), or the group's choice; a single
    // layer gets smaller slices while that is needed to give the GPU ~2048
    // work items
    l.kc4 = slice > 0 ? slice : 8;
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
