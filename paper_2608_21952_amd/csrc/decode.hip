// Single-token decode step on the persistent int8 state: the chunked method with a chunk of one
// token (Sec. 4.2 quantization; Eq. 7-8 chunk state, Eq. 9 state passing, Eq. 10 correction),
// for every (batch, head) at once.  With one token the chunk quantities reduce to
//   cs = dA = dt A,  LUT_state = dt,  q_d = rne(exp(dA) 2^k)
//   X_q[p]    = Q(fl32(dt x[p]) / a_X[p])                          (Eq. 7)
//   S_q[p,n]  = requant(X_q[p] B_q[n], m_S[p])                       (Eq. 8)
//   state'    = sat(S_q + ((q_d state + r) >> k))                    (Eq. 9)
//   y[p]      = (sum_n C_q[n] state[p,n]) a_C exp(dA) a_S[p]         (ChunkScan1, entering state)
//             + fp16(CB_q a_CB dt) fp16(x[p])                        (ChunkScan2, i = j)
//             + D x[p] + corr[p]
// with CB_q = requant(C_q . B_q, m_CB).  Every integer quantity and every fp32 rounding before
// an integer decision is formed exactly as in the chunked kernels (ChunkState, ChunkBMM, state
// passing), so a decode step equals the layer run over that token with chunk size 1.
//
// One workgroup per (b, h), 256 threads: thread t owns state row p = t / 4 and the 32 state
// entries n in [32 (t % 4), +32): one 32-byte read and write of the row-major state, in place.
#include "common.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

template <typename XT, typename YT>
__global__ __launch_bounds__(256) void decode_kernel(
    const XT* __restrict__ x, const float* __restrict__ dt, int dt_softplus,
    const float* __restrict__ A, const int8_t* __restrict__ Bq, const int8_t* __restrict__ Cq,
    const float* __restrict__ B_scale, const float* __restrict__ C_scale, int c_per_token,
    const float* __restrict__ Dv, const float* __restrict__ corr,
    const float* __restrict__ xs_scale, int xs_per_head, const float* __restrict__ state_scale,
    const float* __restrict__ cb_scale, int shift, int radd, int8_t* __restrict__ state,
    YT* __restrict__ y, float* __restrict__ state_f32, int H, int G) {
  const int t = threadIdx.x;
  const int p = t >> 2, n0 = 32 * (t & 3);
  const int bh = blockIdx.x;
  const int b = bh / H, h = bh - b * H;
  const int g = h / (H / G);

  // ---- every load first (none depends on another), then the dependent fp64 chain
  const size_t bg = (size_t)b * G + g;
  const uint4* brow = reinterpret_cast<const uint4*>(Bq + bg * kN + n0);
  const uint4* crow = reinterpret_cast<const uint4*>(Cq + bg * kN + n0);
  uint4* srow = reinterpret_cast<uint4*>(state + ((size_t)bh * kP + p) * kN + n0);
  const uint4 bv[2] = {brow[0], brow[1]};
  const uint4 cv[2] = {crow[0], crow[1]};
  const uint4 sv[2] = {srow[0], srow[1]};
  float dtv = dt[bh];
  const float Ah = A[h];
  const float xval = (float)x[(size_t)bh * kP + p];
  const float axs = xs_per_head ? xs_scale[h] : xs_scale[h * kP + p];
  const float aS = state_scale[h * kP + p];
  const float aB = B_scale[g];

  // ---- the one-token chunk: dt, dA, Q(Decay) (fp64 as in ChunkState)
  if (dt_softplus) dtv = softplus_f32(dtv);
  const float dA = dtv * Ah;
  const double cs = (double)dA;
  const int qd = (int)rint(exp(cs) * (double)(1 << shift));
  const float lut = dtv * (float)exp(cs - cs);

  // ---- X_q of channel p and its state multiplier (Eq. 7-8)
  const float inv = 1.0f / axs;
  const int xq = quant_i8(lut * xval, inv);
  const float ms = (float)(((double)axs * (double)aB) / (double)aS);
  int y1 = 0, cb = 0;
  uint4 nv[2];
  int nf[32];
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    const uint32_t bw[4] = {bv[half].x, bv[half].y, bv[half].z, bv[half].w};
    const uint32_t cw[4] = {cv[half].x, cv[half].y, cv[half].z, cv[half].w};
    const uint32_t sw[4] = {sv[half].x, sv[half].y, sv[half].z, sv[half].w};
    uint32_t ow[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      int o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int bq = sext8(bw[d], e), cq = sext8(cw[d], e), s = sext8(sw[d], e);
        y1 += __mul24(cq, s);               // ChunkScan1 on the entering state
        cb += __mul24(cq, bq);              // C.B^T of the token with itself
        const int sq = requant_i8(__mul24(xq, bq), ms);
        o[e] = pass_step(s, sq, qd, shift, radd);
        nf[16 * half + 4 * d + e] = o[e];
      }
      ow[d] = pack4_i8(o[0], o[1], o[2], o[3]);
    }
    nv[half] = make_uint4(ow[0], ow[1], ow[2], ow[3]);
  }
  // the 4 threads of row p are adjacent lanes
  y1 += __shfl_xor(y1, 1, 64);
  y1 += __shfl_xor(y1, 2, 64);
  cb += __shfl_xor(cb, 1, 64);
  cb += __shfl_xor(cb, 2, 64);
  srow[0] = nv[0];
  srow[1] = nv[1];
  if (state_f32) {
    float4* fo = reinterpret_cast<float4*>(state_f32 + ((size_t)bh * kP + p) * kN + n0);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      fo[u] = make_float4((float)nf[4 * u] * aS, (float)nf[4 * u + 1] * aS,
                          (float)nf[4 * u + 2] * aS, (float)nf[4 * u + 3] * aS);
  }

  if ((t & 3) == 0) {
    const float ac = c_per_token ? C_scale[bg] : C_scale[g];
    const float mcb = (float)(((double)ac * (double)aB) / (double)cb_scale[g]);
    const int cbq = requant_i8(cb, mcb);
    const float dtcb = cb_scale[g] * dtv;
    const _Float16 w = (_Float16)((float)cbq * dtcb);        // W of the diagonal, exp(0) = 1
    const float Dh = Dv ? Dv[h] : 0.0f;
    const float cr = corr ? corr[h * kP + p] : 0.0f;
    float yd = __builtin_fmaf(Dh, xval, cr);
    yd += (float)w * (float)(_Float16)xval;
    const float eo = ac * __expf(dA);
    const float out = __builtin_fmaf((float)y1 * eo, aS, yd);
    y[(size_t)bh * kP + p] = (YT)out;
  }
}

}  // namespace

hipError_t launch_decode(int64_t batch, int64_t nheads, int64_t ngroups, const void* x,
                         int x_dtype, const float* dt, int dt_softplus, const float* A,
                         const int8_t* Bq, const int8_t* Cq, const float* B_scale,
                         const float* C_scale, int c_per_token, const float* D,
                         const float* corr, const float* xs_scale, int xs_per_head,
                         const float* state_scale, const float* cb_scale, int shift,
                         int shift_round, int8_t* state, void* y, int y_dtype, float* state_f32,
                         hipStream_t st) {
  const int64_t nwg = batch * nheads;
  if (nwg == 0) return hipSuccess;
  const int radd = shift_round ? (1 << (shift - 1)) : 0;
#define SSDI8_DECODE_LAUNCH(XT, YT)                                                           \
  hipLaunchKernelGGL((decode_kernel<XT, YT>), dim3((unsigned)nwg), dim3(256), 0, st,          \
                     static_cast<const XT*>(x), dt, dt_softplus, A, Bq, Cq, B_scale, C_scale, \
                     c_per_token, D, corr, xs_scale, xs_per_head, state_scale, cb_scale,      \
                     shift, radd, state, static_cast<YT*>(y), state_f32, (int)nheads,         \
                     (int)ngroups)
  if (x_dtype == 1 && y_dtype == 1) SSDI8_DECODE_LAUNCH(_Float16, _Float16);
  else if (x_dtype == 1) SSDI8_DECODE_LAUNCH(_Float16, float);
  else if (y_dtype == 1) SSDI8_DECODE_LAUNCH(float, _Float16);
  else SSDI8_DECODE_LAUNCH(float, float);
#undef SSDI8_DECODE_LAUNCH
  return hipGetLastError();
}

}  // namespace ssdi8
