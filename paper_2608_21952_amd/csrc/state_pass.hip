// INT8 StatePassing (Eq. 9; Alg. 2 module 3):
//   P_in[0] = init;  P_in[c+1] = clamp(S_q[c] + ((q_d[c] P_in[c] + r) >> k), -127, 127)
// The recurrence is sequential in c but independent per (batch, head, p, n) element, so each
// thread owns 16 (or 4) consecutive int8 elements of one (b, h) slab and walks the chunks.  The
// loads of S_q and q_d do not depend on the running state, so they are issued in batches of
// kDepth chunks, one batch ahead of the dependent integer updates: the kernel is bound by HBM
// bandwidth (read S_q, write P_in), not by the length of the chain.
//
// Inside the SSD layer S_q and P_in are in the MFMA fragment order of frag.hpp (elementwise
// work does not care); the initial state, the final states and the optional P_in tap are
// row-major [p][n], reached through the inverse of that order.
#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

// kW dwords (4 kW int8 elements) per thread; kFragK = 0: S_q / P_in row-major, kFragK = N:
// kslice order with K = N.
template <int kW> struct Vec;
template <> struct Vec<1> {
  static __device__ __forceinline__ void load(const int8_t* p, uint32_t* v) {
    v[0] = *reinterpret_cast<const uint32_t*>(p);
  }
  static __device__ __forceinline__ void store(int8_t* p, const uint32_t* v) {
    *reinterpret_cast<uint32_t*>(p) = v[0];
  }
};
template <> struct Vec<4> {
  static __device__ __forceinline__ void load(const int8_t* p, uint32_t* v) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
  }
  static __device__ __forceinline__ void store(int8_t* p, const uint32_t* v) {
    *reinterpret_cast<uint4*>(p) = make_uint4(v[0], v[1], v[2], v[3]);
  }
};

template <int kDepth, int kW, int kFragK>
__global__ __launch_bounds__(256) void state_pass_kernel(
    const int8_t* __restrict__ sq, const int16_t* __restrict__ qd, int shift, int radd,
    const int8_t* __restrict__ init, int8_t* __restrict__ pin, int8_t* __restrict__ pin_tap,
    int8_t* __restrict__ final_q, float* __restrict__ final_state,
    const float* __restrict__ state_scale, int nc, int H, int64_t elems, int64_t headdim,
    int64_t nthreads) {
  constexpr int kE = 4 * kW;
  const int64_t gt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gt >= nthreads) return;
  const int64_t e = gt * kE;
  const int64_t bh = e / elems;
  const int64_t off = e - bh * elems;   // storage offset of S_q / P_in
  const int64_t b = bh / H, h = bh - b * H;
  int64_t roff = off;                   // row-major offset of the same elements (consecutive)
  if constexpr (kFragK != 0) {
    int row, k;
    frag::kslice_coords((size_t)off, kFragK, &row, &k);
    roff = (int64_t)row * kFragK + k;
  }
  int st[kE];
  if (init) {
    uint32_t v[kW];
    Vec<kW>::load(init + bh * elems + roff, v);
#pragma unroll
    for (int i = 0; i < kE; ++i) st[i] = sext8(v[i >> 2], i & 3);
  } else {
#pragma unroll
    for (int i = 0; i < kE; ++i) st[i] = 0;
  }
  const size_t cstride = (size_t)H * elems;
  const size_t base = ((size_t)b * nc * H + h) * elems + off;
  const int16_t* qrow = qd + bh * nc;
  // batches of kDepth chunks; the loads of batch k+1 are issued before batch k is processed,
  // so a long chunk sequence streams instead of waiting one load latency per batch
  uint32_t v[2][kDepth][kW];
  int q[2][kDepth];
  auto load_batch = [&](int c0, int buf) {
#pragma unroll
    for (int k = 0; k < kDepth; ++k) {
      if (c0 + k < nc) {
        Vec<kW>::load(sq + base + (size_t)(c0 + k) * cstride, v[buf][k]);
        q[buf][k] = qrow[c0 + k];
      }
    }
  };
  auto run_batch = [&](int c0, int buf) {
#pragma unroll
    for (int k = 0; k < kDepth; ++k) {
      if (c0 + k < nc) {
        uint32_t o[kW];
#pragma unroll
        for (int u = 0; u < kW; ++u)
          o[u] = pack4_i8(st[4 * u], st[4 * u + 1], st[4 * u + 2], st[4 * u + 3]);
        Vec<kW>::store(pin + base + (size_t)(c0 + k) * cstride, o);
        if (pin_tap) Vec<kW>::store(pin_tap + base - off + roff + (size_t)(c0 + k) * cstride, o);
#pragma unroll
        for (int i = 0; i < kE; ++i)
          st[i] = pass_step(st[i], sext8(v[buf][k][i >> 2], i & 3), q[buf][k], shift, radd);
      }
    }
  };
  if (nc > 0) load_batch(0, 0);
  for (int c0 = 0; c0 < nc; c0 += 2 * kDepth) {
    if (c0 + kDepth < nc) load_batch(c0 + kDepth, 1);
    run_batch(c0, 0);
    if (c0 + kDepth < nc) {
      if (c0 + 2 * kDepth < nc) load_batch(c0 + 2 * kDepth, 0);
      run_batch(c0 + kDepth, 1);
    }
  }
  if (final_q) {
    uint32_t o[kW];
#pragma unroll
    for (int u = 0; u < kW; ++u)
      o[u] = pack4_i8(st[4 * u], st[4 * u + 1], st[4 * u + 2], st[4 * u + 3]);
    Vec<kW>::store(final_q + bh * elems + roff, o);
  }
  if (final_state) {
    // the kE elements share p when (elems / headdim) % kE == 0 (checked by the launcher)
    const int64_t p = roff / (elems / headdim);
    const float a = state_scale[h * headdim + p];
    float4* fo = reinterpret_cast<float4*>(final_state + bh * elems + roff);
#pragma unroll
    for (int u = 0; u < kW; ++u)
      fo[u] = make_float4((float)st[4 * u] * a, (float)st[4 * u + 1] * a,
                          (float)st[4 * u + 2] * a, (float)st[4 * u + 3] * a);
  }
}

// One 16-byte lane slice of a permuted-kslice P x N slab per thread: row p = 32 (tile / 4) +
// lane % 32, and four runs of four consecutive n at 32 (tile % 4) + 8 g + 4 (lane / 32).
__global__ __launch_bounds__(256) void pin_tap_kernel(const int8_t* __restrict__ pin,
                                                      int8_t* __restrict__ tap, int64_t nslices) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nslices) return;
  constexpr int64_t kSlab = (int64_t)kP * kN;
  const int64_t slab = i / (kSlab / 16);
  const int off = (int)(i - slab * (kSlab / 16)) * 16;
  const uint4 v = *reinterpret_cast<const uint4*>(pin + slab * kSlab + off);
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  int row, k;
  frag::pk_coords((size_t)off, kN, &row, &k);   // k of byte 0; byte 4 g at k + 8 g
  int8_t* dst = tap + slab * kSlab + (int64_t)row * kN + k;
#pragma unroll
  for (int g = 0; g < 4; ++g) *reinterpret_cast<uint32_t*>(dst + 8 * g) = w[g];
}

}  // namespace

hipError_t launch_pin_tap(const int8_t* pin, int8_t* tap, int64_t nslabs, hipStream_t st) {
  const int64_t nslices = nslabs * ((int64_t)kP * kN / 16);
  if (nslices == 0) return hipSuccess;
  hipLaunchKernelGGL(pin_tap_kernel, dim3((unsigned)((nslices + 255) / 256)), dim3(256), 0, st,
                     pin, tap, nslices);
  return hipGetLastError();
}

hipError_t launch_state_pass(int64_t batch, int64_t nchunks, int64_t nheads, int64_t elems,
                             int64_t headdim, const int8_t* sq, const int16_t* qd, int shift,
                             int shift_round, const int8_t* init, int8_t* pin, int8_t* pin_tap,
                             int8_t* final_q, float* final_state, const float* state_scale,
                             int frag_k, hipStream_t st) {
  if (batch * nheads * elems == 0) return hipSuccess;
  const int radd = shift_round ? (1 << (shift - 1)) : 0;
  // 16 elements per thread when a state row holds a multiple of 16 (they then share p) and that
  // still leaves at least 4 waves per CU; else 4 (long sequences of few heads are issue-bound:
  // every thread walks all chunks)
  const bool wide = (elems / headdim) % 16 == 0 && batch * nheads * elems / 16 >= 65536;
  const int64_t nthreads = batch * nheads * elems / (wide ? 16 : 4);
  const unsigned blocks = (unsigned)((nthreads + 255) / 256);
  // short sequences: one batch of 8 chunks covers them; long ones keep 2 x 16 chunks in flight
  const bool deep = nchunks > 8;
#define SSDI8_PASS_LAUNCH(D, W, FK)                                                            \
  hipLaunchKernelGGL((state_pass_kernel<D, W, FK>), dim3(blocks), dim3(256), 0, st, sq, qd,     \
                     shift, radd, init, pin, pin_tap, final_q, final_state, state_scale,        \
                     (int)nchunks, (int)nheads, elems, headdim, nthreads)
  if (frag_k == kN && elems == (int64_t)kP * kN && headdim == kP) {
    if (!wide) SSDI8_PASS_LAUNCH(8, 1, kN);
    else if (deep) SSDI8_PASS_LAUNCH(16, 4, kN);
    else SSDI8_PASS_LAUNCH(8, 4, kN);
  } else if (frag_k == 0) {
    if (wide) SSDI8_PASS_LAUNCH(8, 4, 0);
    else SSDI8_PASS_LAUNCH(8, 1, 0);
  } else {
    return hipErrorInvalidValue;
  }
#undef SSDI8_PASS_LAUNCH
  return hipGetLastError();
}

}  // namespace ssdi8
