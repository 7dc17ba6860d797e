// ChunkCumsum + reformulated INT8 ChunkState (Alg. 2 modules 1-2; Eq. 7-8; Q(Decay) of Eq. 9).
//
// One workgroup per (batch, chunk, head), 256 threads = one thread per token of the chunk:
//   dt      = softplus(dt_raw) (optional), dA = fl32(dt * A[h])
//   cs_j    = in-chunk inclusive sum of dA in fp64 (exact)
//   LUT_j   = fl32(dt_j * fl32(exp(cs_last - cs_j)))                         (Eq. 4 table)
//   X_q     = clamp(rne(fl32(LUT_j * x_jp) * fl32(1/a_X[p])), -127, 127)      (Eq. 7, the decay
//             moved off B onto x so that both MFMA operands are int8)
//   S32     = X_q^T B_q  (int8 MFMA over the 256 tokens, int32 accumulation)
//   S_q     = clamp(rne(fl32(S32) * m_S[p]))  with m_S = fl32(a_X a_B / a_S)   (Eq. 8)
//   q_d     = rne(exp(cs_last) * 2^k)                                          (Eq. 9)
// The contraction runs over tokens, which are strided in HBM: x is loaded row-coalesced (32
// lanes cover one 128-byte token row), quantized in registers and written to LDS already
// transposed ([p][j], tokens contiguous = the MFMA K-slice); B_q^T comes pre-transposed from
// the ChunkBMM kernel in fragment order (frag.hpp).  S_q leaves through an LDS stage in the
// fragment order in which ChunkScan1 reads the entering state (state passing is elementwise, so
// it keeps that order); the optional S_q / S32 taps are row-major [p][n].
#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kXS = kQ + 16;  // LDS row stride (bytes) of X_q^T

// Two adjacent channels of one token row, loaded raw (the loads are issued before the decay table
// they are scaled by is ready) and unpacked to fp32 later.
template <typename XT> struct Pair;
template <> struct Pair<_Float16> {
  typedef uint32_t raw;
  static __device__ __forceinline__ raw load(const _Float16* p) {
    return *reinterpret_cast<const uint32_t*>(p);
  }
  static __device__ __forceinline__ float lo(raw v) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(v & 0xffffu));
  }
  static __device__ __forceinline__ float hi(raw v) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(v >> 16));
  }
};
template <> struct Pair<float> {
  typedef float2 raw;
  static __device__ __forceinline__ raw load(const float* p) {
    return *reinterpret_cast<const float2*>(p);
  }
  static __device__ __forceinline__ float lo(raw v) { return v.x; }
  static __device__ __forceinline__ float hi(raw v) { return v.y; }
};

// fp16 x: at most 80 VGPRs, six workgroups per CU (a 130M-shaped layer's 1536 chunk items fit
// in one round); the fp32-x form keeps four
template <typename XT>
__global__ __launch_bounds__(256, sizeof(XT) == 2 ? 6 : 4) void chunk_state_kernel(
    const XT* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const int8_t* __restrict__ bqT, const float* __restrict__ B_scale,
    const float* __restrict__ xs_scale, int xs_per_head, const float* __restrict__ state_scale,
    int dt_softplus, int shift, int8_t* __restrict__ sq, int16_t* __restrict__ qd,
    int8_t* __restrict__ xq_tap, int8_t* __restrict__ sq_tap, int32_t* __restrict__ s32_tap,
    float* __restrict__ dt_tap, int L, int H, int G, int nc) {
  __shared__ __attribute__((aligned(16))) int8_t s_xq[kP * kXS];
  __shared__ float s_lut[kQ];
  __shared__ float s_inv[kP];
  __shared__ float s_ms[kP];
  __shared__ double s_scan[kScanScratch];
  __shared__ double s_last;

  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int h = w % H;
  const int bc = w / H;
  const int c = bc % nc;
  const int b = bc / nc;
  const int g = h / (H / G);
  const size_t tok0 = (size_t)b * L + (size_t)c * kQ;
  const size_t HP = (size_t)H * kP;

  // ---- issue the x tile loads first (thread: channel pair (p0, p0+1), tokens
  //      [32 jb, 32 jb + 32)); they overlap the ChunkCumsum below
  const int pp = t & 31, jb = t >> 5, p0 = 2 * pp;
  typename Pair<XT>::raw xr[32];
  {
    const XT* xb = x + (tok0 + (size_t)jb * 32) * HP + (size_t)h * kP + p0;
#pragma unroll
    for (int r = 0; r < 32; ++r) xr[r] = Pair<XT>::load(xb + (size_t)r * HP);
  }

  // ---- ChunkCumsum: token t
  float dtv = dt[(tok0 + t) * H + h];
  if (dt_softplus) dtv = softplus_f32(dtv);
  if (dt_tap) dt_tap[(tok0 + t) * H + h] = dtv;
  const float dA = dtv * A[h];
  const double cs = block_scan_f64_256<true>(dA, s_scan, s_lut);
  if (t == kQ - 1) s_last = cs;
  if (t < kP) {
    const float axs = xs_per_head ? xs_scale[h] : xs_scale[h * kP + t];
    s_inv[t] = 1.0f / axs;
    s_ms[t] = (float)(((double)axs * (double)B_scale[g]) / (double)state_scale[h * kP + t]);
  }
  __syncthreads();
  const double last = s_last;
  s_lut[t] = dtv * (float)exp(last - cs);
  if (t == 0) qd[((size_t)b * H + h) * nc + c] = (int16_t)rint(exp(last) * (double)(1 << shift));
  __syncthreads();

  // ---- X_scaled -> X_q, written transposed to LDS ([p][j], tokens contiguous)
  {
    const float inv0 = s_inv[p0], inv1 = s_inv[p0 + 1];
    // quantized and packed 4 token rows at a time, so that the raw rows die as they are used
    uint32_t w0[8], w1[8];
#pragma unroll
    for (int r4 = 0; r4 < 8; ++r4) {
      uint32_t qa[4], qb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * r4 + i;
        const float lut = s_lut[jb * 32 + r];
        // fl32(lut x) as an fma with +0 (for fp16 x, one mixed-precision fma)
        qa[i] = quant_bits(__builtin_fmaf(Pair<XT>::lo(xr[r]), lut, 0.0f), inv0);
        qb[i] = quant_bits(__builtin_fmaf(Pair<XT>::hi(xr[r]), lut, 0.0f), inv1);
      }
      w0[r4] = pack_lo4(qa[0], qa[1], qa[2], qa[3]);
      w1[r4] = pack_lo4(qb[0], qb[1], qb[2], qb[3]);
    }
    int8_t* r0 = s_xq + p0 * kXS + jb * 32;
    int8_t* r1 = r0 + kXS;
    *reinterpret_cast<uint4*>(r0) = make_uint4(w0[0], w0[1], w0[2], w0[3]);
    *reinterpret_cast<uint4*>(r0 + 16) = make_uint4(w0[4], w0[5], w0[6], w0[7]);
    *reinterpret_cast<uint4*>(r1) = make_uint4(w1[0], w1[1], w1[2], w1[3]);
    *reinterpret_cast<uint4*>(r1 + 16) = make_uint4(w1[4], w1[5], w1[6], w1[7]);
    if (xq_tap) {
      int8_t* tb = xq_tap + (tok0 + (size_t)jb * 32) * HP + (size_t)h * kP + p0;
#pragma unroll
      for (int r = 0; r < 32; ++r)
        *reinterpret_cast<uint16_t*>(tb + (size_t)r * HP) =
            (uint16_t)(((w0[r >> 2] >> (8 * (r & 3))) & 0xffu) |
                       (((w1[r >> 2] >> (8 * (r & 3))) & 0xffu) << 8));
    }
  }
  __syncthreads();

  // ---- S32 = X_q^T B_q: wave -> p-tile mt (32 rows), n-tiles ntb, ntb + 1
  const int mt = wv & 1, ntb = (wv >> 1) * 2;
  const int8_t* bq = bqT + (((size_t)b * nc + c) * G + g) * (size_t)kN * kQ;
  v16i acc0 = {}, acc1 = {};
  {
    const int8_t* arow = s_xq + (mt * 32 + (lane & 31)) * kXS;
    // B_q^T fragments of n-tiles ntb, ntb + 1: 1 KB per (n-tile, 32-token block), lane-major
    const int8_t* b0f = bq + (size_t)ntb * (kQ / 32) * 1024 + lane * 16;
    const int8_t* b1f = b0f + (size_t)(kQ / 32) * 1024;
#pragma unroll 4
    for (int ks = 0; ks < kQ / 32; ++ks) {
      const int kof = ks * 32 + 16 * (lane >> 5);
      const v4i a = *reinterpret_cast<const v4i*>(arow + kof);
      const v4i b0 = *reinterpret_cast<const v4i*>(b0f + ks * 1024);
      const v4i b1 = *reinterpret_cast<const v4i*>(b1f + ks * 1024);
      acc0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b1, acc1, 0, 0, 0);
    }
  }
  __syncthreads();  // X_q^T no longer read: its LDS is reused to stage S_q

  // ---- requantize (Eq. 8) and stage S_q in fragment order
  int8_t* s_stage = s_xq;
  const size_t sbase = (((size_t)b * nc + c) * H + h) * (size_t)kP * kN;
  const int n0 = ntb * 32 + (lane & 31);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int p = mt * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    const float ms = s_ms[p];
    s_stage[frag::kslice_offset(p, n0, kN)] = (int8_t)requant_i8(acc0[r], ms);
    s_stage[frag::kslice_offset(p, n0 + 32, kN)] = (int8_t)requant_i8(acc1[r], ms);
  }
  if (s32_tap) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int p = mt * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      s32_tap[sbase + (size_t)p * kN + n0] = acc0[r];
      s32_tap[sbase + (size_t)p * kN + n0 + 32] = acc1[r];
    }
  }
  __syncthreads();
  uint4* dst = reinterpret_cast<uint4*>(sq + sbase);
  const uint4* src = reinterpret_cast<const uint4*>(s_stage);
  dst[t] = src[t];
  dst[t + 256] = src[t + 256];
  if (sq_tap) {
    // row-major copy: 16 consecutive n of one p are one 16-byte slice of the stage
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int idx = k * 256 + t, p = idx >> 3, n = (idx & 7) * 16;
      *reinterpret_cast<uint4*>(sq_tap + sbase + (size_t)p * kN + n) =
          *reinterpret_cast<const uint4*>(s_stage + frag::kslice_offset(p, n, kN));
    }
  }
}

}  // namespace

hipError_t launch_chunk_state(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                              int dt_softplus, const float* A, const int8_t* bqT,
                              const float* B_scale, const float* xs_scale, int xs_per_head,
                              const float* state_scale, int shift, int8_t* sq, int16_t* qd,
                              int8_t* xq_tap, int8_t* sq_tap, int32_t* s32_tap, float* dt_tap,
                              hipStream_t st) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.nheads;
  if (nwork == 0) return hipSuccess;
  if (x_dtype == 1) {
    hipLaunchKernelGGL(chunk_state_kernel<_Float16>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const _Float16*>(x), dt, A, bqT, B_scale, xs_scale,
                       xs_per_head, state_scale, dt_softplus, shift, sq, qd, xq_tap, sq_tap,
                       s32_tap, dt_tap, d.seqlen, d.nheads, d.ngroups, d.nchunks);
  } else {
    hipLaunchKernelGGL(chunk_state_kernel<float>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const float*>(x), dt, A, bqT, B_scale, xs_scale, xs_per_head,
                       state_scale, dt_softplus, shift, sq, qd, xq_tap, sq_tap, s32_tap, dt_tap,
                       d.seqlen, d.nheads, d.ngroups, d.nchunks);
  }
  return hipGetLastError();
}

}  // namespace ssdi8
