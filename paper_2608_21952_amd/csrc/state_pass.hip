// INT8 StatePassing (Eq. 9; Alg. 2 module 3):
//   P_in[0] = init;  P_in[c+1] = clamp(S_q[c] + ((q_d[c] P_in[c] + r) >> k), -127, 127)
// The recurrence is sequential in c but independent per (batch, head, p, n) element, so each
// thread owns 4 consecutive int8 elements of one (b, h) slab and walks the chunks.  The loads
// of S_q and q_d do not depend on the running state, so they are issued kDepth chunks ahead
// (one batch of independent loads, then the dependent integer updates): the kernel is bound by
// HBM bandwidth (read S_q, write P_in), not by the length of the chain.
//
// Inside the SSD layer S_q and P_in are in the MFMA fragment order of frag.hpp (elementwise
// work does not care); the initial state, the final states and the optional P_in tap are
// row-major [p][n], reached through the inverse of that order.
#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

__device__ __forceinline__ int step_state(int s, int add, int q, int shift, int radd) {
  const int v = add + ((q * s + radd) >> shift);
  return v < -kQMax ? -kQMax : (v > kQMax ? kQMax : v);
}

template <int kDepth>
__global__ __launch_bounds__(256) void state_pass_kernel(
    const int8_t* __restrict__ sq, const int16_t* __restrict__ qd, int shift, int radd,
    const int8_t* __restrict__ init, int8_t* __restrict__ pin, int8_t* __restrict__ pin_tap,
    int8_t* __restrict__ final_q, float* __restrict__ final_state,
    const float* __restrict__ state_scale, int nc, int H, int64_t elems, int64_t headdim,
    int frag_k, int64_t nthreads) {
  const int64_t gt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gt >= nthreads) return;
  const int64_t e = gt * 4;
  const int64_t bh = e / elems;
  const int64_t off = e - bh * elems;   // storage offset of S_q / P_in
  const int64_t b = bh / H, h = bh - b * H;
  int64_t roff = off;                   // row-major offset of the same 4 elements
  if (frag_k) {
    int row, k;
    frag::kslice_coords((size_t)off, frag_k, &row, &k);
    roff = (int64_t)row * frag_k + k;
  }
  int s0 = 0, s1 = 0, s2 = 0, s3 = 0;
  if (init) {
    const uint32_t v = *reinterpret_cast<const uint32_t*>(init + bh * elems + roff);
    s0 = sext8(v, 0); s1 = sext8(v, 1); s2 = sext8(v, 2); s3 = sext8(v, 3);
  }
  const size_t cstride = (size_t)H * elems;
  const size_t base = ((size_t)b * nc * H + h) * elems + off;
  const int16_t* qrow = qd + bh * nc;
  for (int c0 = 0; c0 < nc; c0 += kDepth) {
    uint32_t v[kDepth];
    int q[kDepth];
#pragma unroll
    for (int k = 0; k < kDepth; ++k) {
      if (c0 + k < nc) {
        v[k] = *reinterpret_cast<const uint32_t*>(sq + base + (size_t)(c0 + k) * cstride);
        q[k] = qrow[c0 + k];
      }
    }
#pragma unroll
    for (int k = 0; k < kDepth; ++k) {
      if (c0 + k < nc) {
        *reinterpret_cast<uint32_t*>(pin + base + (size_t)(c0 + k) * cstride) =
            pack4_i8(s0, s1, s2, s3);
        if (pin_tap)
          *reinterpret_cast<uint32_t*>(pin_tap + base - off + roff + (size_t)(c0 + k) * cstride) =
              pack4_i8(s0, s1, s2, s3);
        s0 = step_state(s0, sext8(v[k], 0), q[k], shift, radd);
        s1 = step_state(s1, sext8(v[k], 1), q[k], shift, radd);
        s2 = step_state(s2, sext8(v[k], 2), q[k], shift, radd);
        s3 = step_state(s3, sext8(v[k], 3), q[k], shift, radd);
      }
    }
  }
  if (final_q)
    *reinterpret_cast<uint32_t*>(final_q + bh * elems + roff) = pack4_i8(s0, s1, s2, s3);
  if (final_state) {
    const int64_t p = roff / (elems / headdim);
    const float a = state_scale[h * headdim + p];
    // the 4 elements share p when (elems / headdim) % 4 == 0 (checked by the host)
    float4 f = make_float4((float)s0 * a, (float)s1 * a, (float)s2 * a, (float)s3 * a);
    *reinterpret_cast<float4*>(final_state + bh * elems + roff) = f;
  }
}

}  // namespace

hipError_t launch_state_pass(int64_t batch, int64_t nchunks, int64_t nheads, int64_t elems,
                             int64_t headdim, const int8_t* sq, const int16_t* qd, int shift,
                             int shift_round, const int8_t* init, int8_t* pin, int8_t* pin_tap,
                             int8_t* final_q, float* final_state, const float* state_scale,
                             int frag_k, hipStream_t st) {
  const int64_t nthreads = batch * nheads * elems / 4;
  if (nthreads == 0) return hipSuccess;
  const int radd = shift_round ? (1 << (shift - 1)) : 0;
  const unsigned blocks = (unsigned)((nthreads + 255) / 256);
  hipLaunchKernelGGL(state_pass_kernel<16>, dim3(blocks), dim3(256), 0, st, sq, qd, shift, radd,
                     init, pin, pin_tap, final_q, final_state, state_scale, (int)nchunks,
                     (int)nheads, elems, headdim, frag_k, nthreads);
  return hipGetLastError();
}

}  // namespace ssdi8
