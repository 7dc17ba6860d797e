// Exact summation of fp32 values rounded once to fp64, shared by the kernels (the rare path of
// their in-chunk prefix sums) and a host-side check; plain C++ apart from the HIP qualifiers.
#pragma once

#include <stdint.h>

#include <cmath>

#if defined(__HIPCC__)
#define SSDI8_HD __host__ __device__ __forceinline__
#else
#define SSDI8_HD inline
#endif

namespace ssdi8 {

// Fixed point over 2^-149: a finite fp32 value is m 2^(s - 149) with an integer m < 2^24 and
// 0 <= s <= 253, so signed sums of up to 2^33 of them fit 320 bits.  Words are little-endian
// uint64; every index into them is a compile-time constant (unrolled selects), which keeps them
// in registers on the GPU.
constexpr int kFixWords = 5;

// acc += m 2^s, or acc -= m 2^s with `sub` (two's complement over 320 bits).
SSDI8_HD void fix_add(uint64_t (&acc)[kFixWords], uint32_t m, int s, bool sub) {
  const int w = s >> 6, o = s & 63;
  const uint64_t lo = (uint64_t)m << o;
  const uint64_t hi = o > 40 ? (uint64_t)m >> (64 - o) : 0u;
  uint64_t c = 0;   // carry, or borrow
  for (int k = 0; k < kFixWords; ++k) {
    const uint64_t x = k == w ? lo : (k == w + 1 ? hi : 0u);
    const uint64_t a = acc[k];
    if (sub) {
      const uint64_t s1 = a - x, s2 = s1 - c;
      c = (uint64_t)(a < x) | (uint64_t)(s1 < c);
      acc[k] = s2;
    } else {
      const uint64_t s1 = a + x, s2 = s1 + c;
      c = (uint64_t)(s1 < x) | (uint64_t)(s2 < s1);
      acc[k] = s2;
    }
  }
}

// 64 bits of the fixed-point magnitude starting at bit `pos` (0 <= pos < 320).
SSDI8_HD uint64_t fix_bits(const uint64_t (&a)[kFixWords], int pos) {
  const int w = pos >> 6, o = pos & 63;
  uint64_t lo = 0, hi = 0;
  for (int k = 0; k < kFixWords; ++k) {
    if (k == w) lo = a[k];
    if (k == w + 1) hi = a[k];
  }
  return o ? (lo >> o) | (hi << (64 - o)) : lo;
}

// Whether any bit below `pos` (0 <= pos <= 320) is set.
SSDI8_HD bool fix_any_below(const uint64_t (&a)[kFixWords], int pos) {
  bool any = false;
  for (int k = 0; k < kFixWords; ++k) {
    const int b0 = 64 * k;
    if (pos >= b0 + 64) any = any || a[k] != 0u;
    else if (pos > b0) any = any || (a[k] & ((~(uint64_t)0) >> (64 - (pos - b0)))) != 0u;
  }
  return any;
}

// The sum of v[0 .. n) computed exactly and rounded once to fp64 (to nearest, ties to even).
// The terms accumulate in fixed point (two's complement); the magnitude of the total is rounded
// from its leading 53 bits, the next bit and whether any bit below it is set.  A
// non-finite term makes the result the plain fp64 sum (inf or NaN, as IEEE addition gives).
SSDI8_HD double exact_sum_f32(const float* v, int n) {
  uint64_t d[kFixWords] = {0, 0, 0, 0, 0};
  bool finite = true;
  double plain = 0.0;
  for (int i = 0; i < n; ++i) {
    float f = v[i];
    uint32_t b;
    __builtin_memcpy(&b, &f, 4);
    const uint32_t e = (b >> 23) & 0xffu, frac = b & 0x7fffffu;
    plain += (double)f;
    if (e == 0xffu) {
      finite = false;
      continue;
    }
    const uint32_t m = e ? (frac | 0x800000u) : frac;
    if (m != 0u) fix_add(d, m, e ? (int)e - 1 : 0, (b >> 31) != 0u);
  }
  if (!finite) return plain;
  // the sign, then the magnitude
  const bool negative = (d[kFixWords - 1] >> 63) != 0u;
  if (negative) {
    uint64_t c = 1;
    for (int k = 0; k < kFixWords; ++k) {
      const uint64_t x = ~d[k];
      d[k] = x + c;
      c = (uint64_t)(d[k] < c);
    }
  }
  int top = -1;   // index of the leading set bit
  for (int k = 0; k < kFixWords; ++k)
    if (d[k] != 0u) top = 64 * k + 63 - __builtin_clzll(d[k]);
  if (top < 0) return 0.0;
  double r;
  if (top <= 52) {
    r = std::ldexp((double)d[0], -149);   // below 2^53: exact
  } else {
    const int sh = top - 52;
    uint64_t mant = fix_bits(d, sh) & ((((uint64_t)1) << 53) - 1u);
    const bool guard = ((fix_bits(d, sh - 1) & 1u) != 0u);
    const bool sticky = fix_any_below(d, sh - 1);
    if (guard && (sticky || (mant & 1u))) ++mant;   // to nearest, ties to even (2^53 is exact)
    r = std::ldexp((double)mant, sh - 149);
  }
  return negative ? -r : r;
}

}  // namespace ssdi8
