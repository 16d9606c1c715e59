// Device-side pieces shared by the two decode translation units: the
// int8 matrix-core kernels (decode.hip) and the fp8 x fp4 matrix-core
// kernels (decode_f4.hip).  Scalar-register operand loads, layer
// descriptors, buffer resources, the activation operand's layout and the
// streaming ring's cursors and work-item claims.
#pragma once

#include <type_traits>

#include "decode.h"

namespace fairy2i {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

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

// NT consecutive floats (2, 4 or 8) at a wave-uniform address, one scalar load.
// The caller guarantees the NT floats lie inside the allocation.
template <int NT>
__device__ inline void sload_run(const float* p, float (&v)[NT]) {
  if constexpr (NT == 2) {
    sf2 r;
    __asm__ volatile("s_load_dwordx2 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=&s"(r) : "s"(p) : "memory");
    v[0] = r[0];
    v[1] = r[1];
  } else if constexpr (NT == 4) {
    sf4 r;
    __asm__ volatile("s_load_dwordx4 %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=&s"(r) : "s"(p) : "memory");
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = r[i];
  } else {
    static_assert(NT == 8, "2, 4 or 8 floats");
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

// First work item whose first 256-code step is at or after step s (items
// cover steps in table order; an item of row block rb and K slice kc of a
// layer starts at step0 + rb nk4 + kc kc4).  total_items when s is past the
// last step.  L is the layer from the table holding step s, or the only
// layer of a single-layer call.
__device__ inline int64_t item_at_step(const DecLayer& L, int64_t s, const DecHeader& h) {
  if (s >= h.total_steps) return h.total_items;
  const int64_t local = s - L.step0;
  const int64_t rb = local / L.nk4;
  const int rem = (int)(local - rb * L.nk4);
  const int kc = (rem + L.kc4 - 1) / L.kc4;  // kc == nkc rolls over into the next row block (or layer)
  return L.item0 + rb * L.nkc + kc;
}

// Layer holding step s (wave-uniform): the last layer whose step0 <= s.
__device__ inline int find_layer_by_step(const DecLayer* tab, int n, int64_t s) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (uniform64(tab[mid].step0) <= s) lo = mid;
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
  o.gsteps = uniform(p->gsteps);
  o.item0 = uniform64(p->item0);
  o.step0 = uniform64(p->step0);
  o.sitem0 = uniform64(p->sitem0);
  o.sstep0 = uniform64(p->sstep0);
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

// Two 16-byte LDS reads and the wait for them, as one unit (see lds_read4).
__device__ inline void lds_read2(uint32_t a0, uint32_t a1, v4i (&x)[2]) {
  __asm__ volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %3\n\ts_waitcnt lgkmcnt(0)"
                   : "=&v"(x[0]), "=&v"(x[1])
                   : "v"(a0), "v"(a1)
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
constexpr int stream_waves(int NS, int XW, int base = kStreamWaves, int unit = 1024) {
  int w = base;
  while (w > 1 && w * NS * XW * unit > 150 * 1024) w /= 2;
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


// Blocks of kernel k that fit on the current device at once.
inline int resident_blocks(const void* k, int threads) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, threads, 0) != hipSuccess || per_cu < 1)
    return 1024;
  return cus * per_cu;
}

}  // namespace

}  // namespace fairy2i
