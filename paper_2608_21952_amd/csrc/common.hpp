// Device helpers shared by the gfx950 kernels of libssdi8.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "exact_sum.hpp"

namespace ssdi8 {

// Fixed problem geometry of the kernels: headdim P, state size N, chunk length Q.
constexpr int kP = 64;
constexpr int kN = 128;
constexpr int kQ = 256;
constexpr int kQMax = 127;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

// Raw buffer resource over the bytes from `base` (gfx9 layout: 48-bit base, stride 0, no range
// limit, dword 3 = 0x00020000).  A buffer access adds a per-lane 32-bit offset and a wave-uniform
// 32-bit offset on the address unit, where a global access needs a 64-bit vector add per
// access.  Callers keep every offset inside the tensor they address.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)0xffffffffu,
                                           0x00020000);
}
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                            uint32_t soff) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}
// Cache policy of a buffer access (gfx950): 0 the default; kPolicyNT non-temporal, for data a
// kernel touches once (streamed through the caches instead of displacing what is reused).
constexpr int kPolicyNT = 2;
template <int kPol = 0>
__device__ __forceinline__ uint2 buf_load8(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                           uint32_t soff) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, kPol);
  return make_uint2(v[0], v[1]);
}
template <int kPol = 0>
__device__ __forceinline__ uint32_t buf_load4(__amdgpu_buffer_rsrc_t r, uint32_t voff,
                                              uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, kPol);
}
template <int kPol = 0>
__device__ __forceinline__ void buf_store16(uint4 d, __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                            uint32_t soff) {
  typedef uint32_t u32x4 __attribute__((vector_size(16)));
  const u32x4 v = {d.x, d.y, d.z, d.w};
  __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)voff, (int)soff, kPol);
}

// Symmetric int8 quantization of an fp32 value with a precomputed inverse step:
// clamp(rne(v * inv), -127, 127).  One IEEE fp32 product, round-half-even to integer.  Formed
// as rne(clamp(p)), which is the same value (rne is monotonic and fixes +-127), with the
// rounding done by adding 1.5 * 2^23: every sum lies in [2^23, 2^24), where fp32 steps by 1,
// so the addition rounds c to an integer, ties to even, and the sum's bit pattern is
// 0x4B400000 + c; its low byte is c as a two's-complement int8.  A NaN product clamps to -127
// either way.
// quant_bits returns that bit pattern (the code in its low byte), for packing; quant_i8 the code.
__device__ __forceinline__ uint32_t quant_bits(float v, float inv) {
  const float c = __builtin_fminf(__builtin_fmaxf(v * inv, -127.0f), 127.0f);
  return __builtin_bit_cast(uint32_t, c + 12582912.0f);
}
__device__ __forceinline__ int quant_i8(float v, float inv) {
  return (int)quant_bits(v, inv) - 0x4B400000;
}

// INT32 accumulator -> int8 with an fp32 multiplier: clamp(rne(fl32(acc) * m)).
__device__ __forceinline__ uint32_t requant_bits(int acc, float m) {
  return quant_bits((float)acc, m);
}
__device__ __forceinline__ int requant_i8(int acc, float m) {
  return quant_i8((float)acc, m);
}

// One INT8 StatePassing step of an element (Eq. 9): clamp(S_q + ((q_d P_in + r) >> k), +-127)
// with an arithmetic shift.  q_d is an int16 and P_in an int8, so the product is exact in the
// full-rate 24-bit multiply (a plain int product compiles to the quarter-rate 32-bit one).
__device__ __forceinline__ int pass_step(int s, int add, int q, int shift, int radd) {
  const int v = add + ((__mul24(q, s) + radd) >> shift);
  return v < -kQMax ? -kQMax : (v > kQMax ? kQMax : v);
}

// The same step on the four int8 elements of a dword pair (state word p, chunk-local word s),
// two elements per packed 16-bit instruction.  Valid for shift <= 8 with 0 <= q <= 2^shift:
// |q P + r| <= 256 * 127 + 128 < 2^15, so every value fits an int16 and the packed arithmetic
// is exact.  Bytes are sign-extended by a left shift of the dword and arithmetic right shifts
// of its halves (even bytes: (w << 8) >> 8 per half; odd bytes: w >> 8 per half), and the
// results are gathered back with one byte permute.
typedef short s16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pass_step4_pk16(uint32_t p, uint32_t s, s16x2 q, s16x2 r,
                                                    s16x2 shift) {
  const s16x2 eight = {8, 8};
  const s16x2 pe = __builtin_bit_cast(s16x2, p << 8) >> eight;
  const s16x2 po = __builtin_bit_cast(s16x2, p) >> eight;
  const s16x2 se = __builtin_bit_cast(s16x2, s << 8) >> eight;
  const s16x2 so = __builtin_bit_cast(s16x2, s) >> eight;
  const s16x2 lo = {-kQMax, -kQMax}, hi = {kQMax, kQMax};
  s16x2 ve = se + ((q * pe + r) >> shift);
  s16x2 vo = so + ((q * po + r) >> shift);
  ve = __builtin_elementwise_max(__builtin_elementwise_min(ve, hi), lo);
  vo = __builtin_elementwise_max(__builtin_elementwise_min(vo, hi), lo);
  // bytes (ve.x, vo.x, ve.y, vo.y)
  return __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, vo), __builtin_bit_cast(uint32_t, ve),
                               0x06020400u);
}

// The low bytes of four words in one dword (byte i = low byte of w_i): two byte permutes and a
// shift-or.
__device__ __forceinline__ uint32_t pack_lo4(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3) {
  const uint32_t lo = __builtin_amdgcn_perm(w1, w0, 0x0c0c0400u);
  const uint32_t hi = __builtin_amdgcn_perm(w3, w2, 0x0c0c0400u);
  return lo | (hi << 16);
}

// softplus in fp64 with the usual threshold (log1p(exp(v)) for v <= 20, v above), rounded once
// to fp32.  On [-40, 20] a short fp64 evaluation (relative error below 2^-50) is rounded where it
// lies at least 2^-44 (relative) from an fp32 rounding boundary, so it rounds as the exact value
// does; elsewhere, and outside [-40, 20], the library's exp and log1p decide (Ziv's strategy).
// The short form: softplus(d) = max(d, 0) + log1p(z), z = exp(-|d|) in (0, 1], with exp by
// Cody-Waite reduction to |r| <= ln2 / 2 and the degree-12 Taylor polynomial, and
// log1p(z) = log(u) + (z - (u - 1)) / u for u = fl(1 + z) (the second term restores the rounding
// of u), log(u) = e ln2 + 2 atanh(s), s = (m - 1) / (m + 1), m = u 2^-e in (0.707, 1.414], and
// atanh's odd series through s^19 (|s| <= 0.172).
__device__ __forceinline__ float softplus_f32(float v) {
  const double d = (double)v;
  if (d > 20.0) return v;
  bool ok = d >= -40.0;
  float out = 0.0f;
  if (ok) {
    constexpr double kLn2Hi = 6.93147180369123816490e-01;   // 32 significant bits
    constexpr double kLn2Lo = 1.90821492927058770002e-10;
    constexpr double kLog2e = 1.4426950408889634;
    const double x = -__builtin_fabs(d);
    const double k = __builtin_rint(x * kLog2e);
    double r = __builtin_fma(-k, kLn2Hi, x);
    r = __builtin_fma(-k, kLn2Lo, r);
    double p = 1.0 / 479001600.0;                            // 1/12!
    p = __builtin_fma(p, r, 1.0 / 39916800.0);
    p = __builtin_fma(p, r, 1.0 / 3628800.0);
    p = __builtin_fma(p, r, 1.0 / 362880.0);
    p = __builtin_fma(p, r, 1.0 / 40320.0);
    p = __builtin_fma(p, r, 1.0 / 5040.0);
    p = __builtin_fma(p, r, 1.0 / 720.0);
    p = __builtin_fma(p, r, 1.0 / 120.0);
    p = __builtin_fma(p, r, 1.0 / 24.0);
    p = __builtin_fma(p, r, 1.0 / 6.0);
    p = __builtin_fma(p, r, 0.5);
    p = __builtin_fma(p, r, 1.0);
    p = __builtin_fma(p, r, 1.0);
    const double z = __builtin_ldexp(p, (int)k);
    const double u = 1.0 + z;
    const double c = z - (u - 1.0);
    const bool big = u > 1.4142135623730951;
    const double m = big ? u * 0.5 : u;
    const double f = m - 1.0;
    const double den = 2.0 + f;
    double q = __builtin_amdgcn_rcp(den);
    q = __builtin_fma(q, __builtin_fma(-den, q, 1.0), q);
    const double s0 = f * q;
    const double s = __builtin_fma(__builtin_fma(-den, s0, f), q, s0);
    const double t = s * s;
    double P = 2.0 / 19.0;
    P = __builtin_fma(P, t, 2.0 / 17.0);
    P = __builtin_fma(P, t, 2.0 / 15.0);
    P = __builtin_fma(P, t, 2.0 / 13.0);
    P = __builtin_fma(P, t, 2.0 / 11.0);
    P = __builtin_fma(P, t, 2.0 / 9.0);
    P = __builtin_fma(P, t, 2.0 / 7.0);
    P = __builtin_fma(P, t, 2.0 / 5.0);
    P = __builtin_fma(P, t, 2.0 / 3.0);
    const double corr = __builtin_fma(c, __builtin_amdgcn_rcp(u), big ? kLn2Lo : 0.0);
    const double lo = __builtin_fma(s, t * P, corr);
    const double l1p = (big ? kLn2Hi : 0.0) + (2.0 * s + lo);
    const double y = d > 0.0 ? d + l1p : l1p;
    const float y0 = (float)(y * (1.0 - 0x1p-44)), y1 = (float)(y * (1.0 + 0x1p-44));
    ok = y0 == y1;
    out = y0;
  }
  if (!ok) out = (float)log1p(exp(d));
  return out;
}

// Map a linear block id to a work index so that consecutive work items land on the same XCD.
// Workgroups are dispatched round-robin over the 8 XCDs of the chip; this inverts that so
// each XCD owns one contiguous range of work (neighbouring heads of one chunk share B, C and
// CB tiles through that XCD's L2).
__device__ __forceinline__ int xcd_remap(int bid, int nwg) {
  constexpr int kXcd = 8;
  int q = nwg / kXcd, r = nwg % kXcd;
  int xcd = bid % kXcd, idx = bid / kXcd;
  return (xcd < r) ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

// v + the value of the lane that DPP control kCtrl selects (0 where there is none or where the
// lane's row is outside kRowMask): one 64-lane data-parallel-primitive move per 32-bit half.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double dpp_add_f64(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, kCtrl, kRowMask,
                                                            0xf, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), kCtrl,
                                                            kRowMask, 0xf, false);
  return v + __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Packed exponent range of a term for the exactness test of block_scan_f64_256: low half
// e + 256, high half 256 - e, with e the exponent of |v| in [2^(e-1), 2^e); subnormals take
// e = -149 (a lower bound, which only makes the test stricter); zero gives 0, the identity of the
// halfwise max.
__device__ __forceinline__ uint32_t exp_range_f32(float v) {
  const uint32_t b = __float_as_uint(v) & 0x7fffffffu;
  if (b == 0) return 0u;
  const int f = (int)(b >> 23);
  const int e = f ? f - 126 : -149;
  return (uint32_t)(e + 256) | ((uint32_t)(256 - e) << 16);
}
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t max_u16x2(uint32_t a, uint32_t b) {
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2, a),
                                                                __builtin_bit_cast(u16x2, b)));
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_max_u16x2(uint32_t v) {
  return max_u16x2(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kCtrl, kRowMask, 0xf,
                                                            false));
}

// Inclusive prefix sum over the 256 threads of a block of fp32 terms, exact and rounded once to
// fp64.  A tree of fp64 additions gives it when every partial sum is exact: the nonzero terms are
// multiples of 2^(e_min - 24) and every partial sum stays below 2^(e_max + 8), so it holds when
// e_max - e_min <= 21 (e: the exponent of |v| in [2^(e-1), 2^e)).  That is the case the block
// tests for; the tree then runs within a wave as shifts by 1, 2, 4, 8 lanes inside each row of
// 16 (row_shr), the last lane of row 0 / 2 into rows 1 / 3 (row_bcast:15) and the last lane of
// row 1 into rows 2 and 3 (row_bcast:31), all in registers, and across the four waves through
// `scratch`.  A block with a wider range (only inputs far outside the method's domain, e.g. dt
// over 20 binades within one chunk) instead sums each prefix exactly (exact_sum_f32) from `stage`.
// scratch: kScanScratch doubles; stage: 256 floats of LDS that the caller writes only after this
// returns.  Every thread of the block must call it.
// kOutlined: the exact path as a call (for kernels whose registers are tight where they scan; the
// call keeps the rare path's registers out of the rest of the kernel).
constexpr int kScanScratch = 6;
static __device__ __noinline__ double exact_sum_f32_outlined(const float* v, int n) {
  return exact_sum_f32(v, n);
}
template <bool kOutlined = false>
__device__ __forceinline__ double block_scan_f64_256(float term, double* scratch, float* stage) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  double v = (double)term;
  uint32_t er = exp_range_f32(term);
  v = dpp_add_f64<0x111, 0xf>(v);
  v = dpp_add_f64<0x112, 0xf>(v);
  v = dpp_add_f64<0x114, 0xf>(v);
  v = dpp_add_f64<0x118, 0xf>(v);
  v = dpp_add_f64<0x142, 0xa>(v);
  v = dpp_add_f64<0x143, 0xc>(v);
  er = dpp_max_u16x2<0x111, 0xf>(er);
  er = dpp_max_u16x2<0x112, 0xf>(er);
  er = dpp_max_u16x2<0x114, 0xf>(er);
  er = dpp_max_u16x2<0x118, 0xf>(er);
  er = dpp_max_u16x2<0x142, 0xa>(er);
  er = dpp_max_u16x2<0x143, 0xc>(er);
  uint32_t* sr = reinterpret_cast<uint32_t*>(scratch + 4);
  if (lane == 63) {
    scratch[w] = v;
    sr[w] = er;
  }
  __syncthreads();
  const uint32_t r = max_u16x2(max_u16x2(sr[0], sr[1]), max_u16x2(sr[2], sr[3]));
  const int e_max = (int)(r & 0xffffu) - 256, e_min = 256 - (int)(r >> 16);
  if (r == 0u || e_max - e_min <= 21) {
    double pre = 0.0;
    for (int i = 0; i < w; ++i) pre += scratch[i];
    return v + pre;
  }
  stage[threadIdx.x] = term;
  __syncthreads();
  const double cs = kOutlined ? exact_sum_f32_outlined(stage, threadIdx.x + 1)
                              : exact_sum_f32(stage, threadIdx.x + 1);
  __syncthreads();
  return cs;
}

// Pack the low bytes of four ints into one dword (byte i = v_i).
__device__ __forceinline__ uint32_t pack4_i8(int v0, int v1, int v2, int v3) {
  return (uint32_t)(v0 & 0xff) | ((uint32_t)(v1 & 0xff) << 8) | ((uint32_t)(v2 & 0xff) << 16) |
         ((uint32_t)(v3 & 0xff) << 24);
}

__device__ __forceinline__ int sext8(uint32_t w, int byte) {
  return (int)(int8_t)((w >> (8 * byte)) & 0xffu);
}

}  // namespace ssdi8
