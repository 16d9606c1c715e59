// Exact summation of non-negative finite doubles and single rounding of
// their mean to float32.  Used for the axis scales of Eq. (ifairy-scale):
// the scale is the exact group mean rounded once, so it does not depend on
// the order in which the GPU adds the values.
//
// A value v = m * 2^(e) (m < 2^53) is an integer multiple of 2^-1074, the
// smallest subnormal double.  The sum is kept as an integer in units of
// 2^-1074 split into SA_LIMBS limbs of 32 bits, each held in a uint64 so
// that up to 2^31 additions never overflow before the carries are resolved.
#pragma once

#include <stdint.h>

#ifndef FAIRY2I_HD
#define FAIRY2I_HD __host__ __device__
#endif

// Bits 0 .. 2045+84 of the fixed-point sum: 66 limbs of 32 bits.
#define SA_LIMBS 66

// Split non-negative finite v into (limb, three 32-bit chunks) such that
// v / 2^-1074 = lo * 2^(32 limb) + mid * 2^(32 (limb+1)) + hi * 2^(32 (limb+2)).
FAIRY2I_HD inline void sa_split(double v, int* limb, uint32_t* lo, uint32_t* mid, uint32_t* hi) {
  uint64_t bits;
#ifdef __HIP_DEVICE_COMPILE__
  bits = (uint64_t)__double_as_longlong(v);
#else
  __builtin_memcpy(&bits, &v, 8);
#endif
  const int E = (int)((bits >> 52) & 0x7FF);
  uint64_t M = bits & ((1ull << 52) - 1);
  if (E > 0) M |= (1ull << 52);
  const int p = (E > 0 ? E : 1) - 1;  // position of M's lowest bit in units of 2^-1074
  const int sh = p & 31;
  *limb = p >> 5;
  *lo = (uint32_t)(M << sh);
  *mid = (uint32_t)(sh == 0 ? (M >> 32) : (M >> (32 - sh)));
  *hi = (uint32_t)(sh == 0 ? 0 : (M >> (64 - sh)));
}

// Loops over the words run with constant indices (fully unrolled on the
// device), so the words stay in registers: every word a position selects is
// picked by comparison, never by a computed index.
#ifdef __HIP_DEVICE_COMPILE__
#define SA_UNROLL _Pragma("unroll")
#else
#define SA_UNROLL
#endif

// Round (sum of limbs) * 2^-1074 / n to the nearest float32, ties to even.
// `limbs` may be unnormalised (each < 2^63); n >= 1 and n <= 2^31.
FAIRY2I_HD inline float sa_mean_to_f32(const uint64_t* limbs, uint64_t n) {
  uint32_t w[SA_LIMBS + 1];
  uint64_t carry = 0;
  SA_UNROLL
  for (int i = 0; i < SA_LIMBS; ++i) {
    const uint64_t v = limbs[i] + carry;
    w[i] = (uint32_t)v;
    carry = v >> 32;
  }
  w[SA_LIMBS] = (uint32_t)carry;
  int h = -1;  // highest nonzero word
  SA_UNROLL
  for (int i = 0; i <= SA_LIMBS; ++i)
    if (w[i] != 0) h = i;
  if (h < 0) return 0.0f;
  uint32_t wh = 0;
  SA_UNROLL
  for (int i = 0; i <= SA_LIMBS; ++i)
    if (i == h) wh = w[i];
  const int bitlen = 32 * h + (32 - __builtin_clz(wh));
  // S64 = top 64 bits of the sum (bit bitlen-1 becomes bit 63), sticky = any
  // bit below them is set.
  uint64_t S64;
  bool sticky = false;
  int shift = bitlen - 64;  // S = S64 * 2^shift + low bits
  if (shift <= 0) {
    uint64_t S = (uint64_t)w[0] | ((h >= 1 ? (uint64_t)w[1] : 0ull) << 32);
    S64 = S << (-shift);
  } else {
    const int ws = shift >> 5, bs = shift & 31;
    uint32_t a0 = 0, a1 = 0, a2 = 0;  // words ws, ws + 1, ws + 2 (0 past the top)
    SA_UNROLL
    for (int i = 0; i <= SA_LIMBS; ++i) {
      if (i == ws) a0 = w[i];
      if (i == ws + 1) a1 = w[i];
      if (i == ws + 2) a2 = w[i];
      if (i < ws && w[i] != 0) sticky = true;
    }
    const uint64_t lo64 = (uint64_t)a0 | ((uint64_t)a1 << 32);
    const uint64_t top = (uint64_t)a2;
    S64 = bs == 0 ? lo64 : ((lo64 >> bs) | (top << (64 - bs)));
    if (bs != 0 && (a0 & ((1u << bs) - 1u)) != 0) sticky = true;
  }
  // value = (S64 + frac) * 2^shift * 2^-1074 / n = (q + delta) * 2^E
  const uint64_t q = S64 / n;
  const uint64_t r = S64 % n;
  if (r != 0) sticky = true;
  const int E = shift - 1074;
  const int qb = 64 - __builtin_clzll(q);  // q >= 2^32 since S64 >= 2^63, n <= 2^31
  const int ebit = qb - 1 + E;             // value in [2^ebit, 2^(ebit+1))
  const bool subnormal = ebit < -126;
  const int ulp = subnormal ? -149 : ebit - 23;
  const int drop = ulp - E;  // low bits of q below the float32 ulp (>= 9)
  uint64_t mant;
  if (drop > 64) {
    mant = 0;  // below half an ulp of the smallest subnormal
  } else {
    mant = drop == 64 ? 0 : (q >> drop);
    const uint64_t rem = drop == 64 ? q : (q & ((1ull << drop) - 1));
    const uint64_t half = 1ull << (drop - 1);
    if (rem > half || (rem == half && (sticky || (mant & 1)))) mant += 1;
  }
  uint32_t out;
  if (subnormal) {
    out = (uint32_t)mant;  // 2^23 after rounding encodes the smallest normal
  } else {
    const int64_t b = ((int64_t)(ebit + 126) << 23) + (int64_t)mant;
    out = b >= 0x7F800000ll ? 0x7F800000u : (uint32_t)b;
  }
  float f;
#ifdef __HIP_DEVICE_COMPILE__
  f = __uint_as_float(out);
#else
  __builtin_memcpy(&f, &out, 4);
#endif
  return f;
}
