// Static-step calibration and the single-layer mean correction on the device (Sec. 5 setup:
// symmetric static steps from a calibration draw; Eq. 10 / Alg. 1 restricted to one layer).
//   alpha_B, alpha_C   absmax / 127 per group            (the dynamic quantizer, Eq. 1)
//   alpha_Xs           absmax of X_scaled = LUT_state x per (h, p) or per h   (Eq. 7)
//   alpha_S            absmax over (b, c, n) of the chunk-local and the passed fp states,
//                      per (h, p) (Eq. 8: the int8 states must rarely saturate)
//   alpha_CB           absmax of the causal entries of C B^T per group
//   corr[h, p]         eta * mean over (b, l) of (Y_fp - Y_q), Y_q the INT8 layer with corr = 0
// X_scaled is formed with exactly the fp32 operations of ChunkState, so alpha_Xs is exact.  The fp
// states are accumulated from x~ = fl32(LUT x) split into two fp16 parts (hi = fp16(x~),
// lo = fp16(x~ - hi)), about 22 significant bits, times fp16 B, in fp32; C B^T of fp16 C, B is
// exact per product and summed in fp32.  Y_fp is the FP16 layer.
#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kXS = kQ * 2 + 16;

typedef _Float16 h8 __attribute__((ext_vector_type(8)));

template <typename XT> __device__ __forceinline__ float2 load_pair(const XT* p);
template <> __device__ __forceinline__ float2 load_pair<_Float16>(const _Float16* p) {
  const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
  return make_float2((float)__builtin_bit_cast(_Float16, (uint16_t)(v & 0xffffu)),
                     (float)__builtin_bit_cast(_Float16, (uint16_t)(v >> 16)));
}
template <> __device__ __forceinline__ float2 load_pair<float>(const float* p) {
  return *reinterpret_cast<const float2*>(p);
}

// ChunkCumsum of one (b, c, h) item as in ChunkState: LUT_state per token into s_lut, the
// chunk decay exp(cs_last) returned (fp64).
__device__ __forceinline__ double lut_of_chunk(const float* dt, const float* A, int dt_softplus,
                                               size_t tok0, int H, int h, float* s_lut,
                                               double* s_scan, double* s_last) {
  const int t = threadIdx.x;
  float dtv = dt[(tok0 + t) * H + h];
  if (dt_softplus) dtv = softplus_f32(dtv);
  const float dA = dtv * A[h];
  const double cs = block_scan_f64_256(dA, s_scan, s_lut);
  if (t == kQ - 1) *s_last = cs;
  __syncthreads();
  const double last = *s_last;
  s_lut[t] = dtv * (float)exp(last - cs);
  __syncthreads();
  return last;
}

// ---- alpha_Xs: per (b, c, h), the absmax over the chunk's tokens of |fl32(LUT x)| per channel
template <typename XT>
__global__ __launch_bounds__(256) void calib_xs_kernel(const XT* __restrict__ x,
                                                       const float* __restrict__ dt,
                                                       const float* __restrict__ A,
                                                       int dt_softplus,
                                                       uint32_t* __restrict__ xs_amax, int L,
                                                       int H, int nc) {
  __shared__ float s_lut[kQ];
  __shared__ double s_scan[kScanScratch];
  __shared__ double s_last;
  __shared__ float s_m[8][kP];
  const int t = threadIdx.x;
  const int w = blockIdx.x;
  const int h = w % H, bc = w / H, c = bc % nc, b = bc / nc;
  const size_t tok0 = (size_t)b * L + (size_t)c * kQ;
  const size_t HP = (size_t)H * kP;
  lut_of_chunk(dt, A, dt_softplus, tok0, H, h, s_lut, s_scan, &s_last);
  const int pp = t & 31, jb = t >> 5, p0 = 2 * pp;
  float m0 = 0.0f, m1 = 0.0f;
  const XT* xb = x + (tok0 + (size_t)jb * 32) * HP + (size_t)h * kP + p0;
#pragma unroll 8
  for (int r = 0; r < 32; ++r) {
    const float2 v = load_pair<XT>(xb + (size_t)r * HP);
    const float lut = s_lut[jb * 32 + r];
    m0 = __builtin_fmaxf(m0, __builtin_fabsf(lut * v.x));
    m1 = __builtin_fmaxf(m1, __builtin_fabsf(lut * v.y));
  }
  s_m[jb][p0] = m0;
  s_m[jb][p0 + 1] = m1;
  __syncthreads();
  if (t < kP) {
    float m = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) m = __builtin_fmaxf(m, s_m[k][t]);
    atomicMax(xs_amax + h * kP + t, __float_as_uint(m));
  }
}

// ---- fp states of each chunk from the split x~ (two fp16 MFMA products), in the fragment order
//      of the FP16 path, plus the chunk decay exp(cs_last) in fp32 and fp64
template <typename XT>
__global__ __launch_bounds__(256) void calib_state_kernel(
    const XT* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const _Float16* __restrict__ bT_frag, int dt_softplus, float* __restrict__ S,
    double* __restrict__ dec64, int L, int H, int G, int nc) {
  __shared__ __attribute__((aligned(16))) uint8_t s_x[kP * kXS];
  __shared__ float s_lut[kQ];
  __shared__ double s_scan[kScanScratch];
  __shared__ double s_last;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int w = blockIdx.x;
  const int h = w % H, bc = w / H, c = bc % nc, b = bc / nc;
  const int g = h / (H / G);
  const size_t tok0 = (size_t)b * L + (size_t)c * kQ;
  const size_t HP = (size_t)H * kP;
  const double last = lut_of_chunk(dt, A, dt_softplus, tok0, H, h, s_lut, s_scan, &s_last);
  if (t == 0) dec64[((size_t)b * H + h) * nc + c] = exp(last);
  const int pp = t & 31, jb = t >> 5, p0 = 2 * pp;
  // x~ = fl32(LUT x) = hi + lo (+ a remainder below 2^-22 |x~|), both parts as fp16, transposed
  // ([p][j], tokens contiguous); the hi parts go through the LDS first, then the lo parts
  uint32_t h0[16], h1[16], l0[16], l1[16];
  {
    const XT* xb = x + (tok0 + (size_t)jb * 32) * HP + (size_t)h * kP + p0;
#pragma unroll
    for (int r2 = 0; r2 < 16; ++r2) {
      uint16_t hb[2][2], lb[2][2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int r = 2 * r2 + q;
        const float2 v = load_pair<XT>(xb + (size_t)r * HP);
        const float lut = s_lut[jb * 32 + r];
        const float xs[2] = {lut * v.x, lut * v.y};
#pragma unroll
        for (int ch = 0; ch < 2; ++ch) {
          const _Float16 hi = (_Float16)xs[ch];
          const _Float16 lo = (_Float16)(xs[ch] - (float)hi);
          hb[ch][q] = __builtin_bit_cast(uint16_t, hi);
          lb[ch][q] = __builtin_bit_cast(uint16_t, lo);
        }
      }
      h0[r2] = hb[0][0] | ((uint32_t)hb[0][1] << 16);
      h1[r2] = hb[1][0] | ((uint32_t)hb[1][1] << 16);
      l0[r2] = lb[0][0] | ((uint32_t)lb[0][1] << 16);
      l1[r2] = lb[1][0] | ((uint32_t)lb[1][1] << 16);
    }
  }
  const int mt = wv & 1, ntb = (wv >> 1) * 2, half = lane >> 5;
  const _Float16* bq = bT_frag + (((size_t)b * nc + c) * G + g) * (size_t)kN * kQ;
  const int ao = (mt * 32 + (lane & 31)) * kXS + 16 * half;
  const _Float16* b0f = bq + (size_t)ntb * (kQ / 16) * 512 + lane * 8;
  const _Float16* b1f = b0f + (size_t)(kQ / 16) * 512;
  v16f acc0 = {}, acc1 = {};
#pragma unroll
  for (int part = 0; part < 2; ++part) {
    const uint32_t* w0 = part == 0 ? h0 : l0;
    const uint32_t* w1 = part == 0 ? h1 : l1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int o0 = p0 * kXS + jb * 64 + 16 * q;
      *reinterpret_cast<uint4*>(s_x + o0) =
          make_uint4(w0[4 * q], w0[4 * q + 1], w0[4 * q + 2], w0[4 * q + 3]);
      *reinterpret_cast<uint4*>(s_x + o0 + kXS) =
          make_uint4(w1[4 * q], w1[4 * q + 1], w1[4 * q + 2], w1[4 * q + 3]);
    }
    __syncthreads();
#pragma unroll 4
    for (int ks = 0; ks < kQ / 16; ++ks) {
      const h8 a = *reinterpret_cast<const h8*>(s_x + ao + ks * 32);
      const h8 b0 = *reinterpret_cast<const h8*>(b0f + ks * 512);
      const h8 b1 = *reinterpret_cast<const h8*>(b1f + ks * 512);
      acc0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b1, acc1, 0, 0, 0);
    }
    __syncthreads();
  }
  float* s_st = reinterpret_cast<float*>(s_x);
  const int n0 = ntb * 32 + (lane & 31);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int p = mt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
    s_st[frag::k16_offset(p, n0, kN)] = acc0[r];
    s_st[frag::k16_offset(p, n0 + 32, kN)] = acc1[r];
  }
  __syncthreads();
  float4* dst = reinterpret_cast<float4*>(S + (((size_t)b * nc + c) * H + h) * (size_t)kP * kN);
  const float4* src = reinterpret_cast<const float4*>(s_st);
#pragma unroll
  for (int k = 0; k < (kP * kN) / (4 * 256); ++k) dst[k * 256 + t] = src[k * 256 + t];
}

// ---- absmax of the chunk-local states and of the states after each chunk (fp64 passing, as
//      the calibration reference) per (h, p); 4 elements (one p) per thread
__global__ __launch_bounds__(256) void calib_pass_kernel(const float* __restrict__ S,
                                                         const double* __restrict__ dec64,
                                                         uint32_t* __restrict__ s_amax, int nc,
                                                         int H, int64_t nthreads) {
  constexpr int64_t kE = (int64_t)kP * kN;
  const int64_t gt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gt >= nthreads) return;
  const int64_t e = gt * 4;
  const int64_t bh = e / kE;
  const int64_t off = e - bh * kE;
  const int64_t b = bh / H, h = bh - b * H;
  int p, n;
  frag::k16_coords((size_t)off, kN, &p, &n);
  double run[4] = {0.0, 0.0, 0.0, 0.0};
  float m = 0.0f;
  const size_t cstride = (size_t)H * kE;
  const size_t base = ((size_t)b * nc * H + h) * kE + off;
  for (int c = 0; c < nc; ++c) {
    const float4 s = *reinterpret_cast<const float4*>(S + base + (size_t)c * cstride);
    const double d = dec64[bh * nc + c];
    const float sv[4] = {s.x, s.y, s.z, s.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      run[q] = (double)sv[q] + d * run[q];
      m = __builtin_fmaxf(m, __builtin_fmaxf(__builtin_fabsf(sv[q]),
                                             (float)__builtin_fabs(run[q])));
    }
  }
  // the two threads of one fragment lane (4 + 4 columns of row p) are neighbours; every
  // workgroup is whole (the thread count is a multiple of 256), so the shuffle is safe
  m = __builtin_fmaxf(m, __shfl_xor(m, 1, 64));
  if ((threadIdx.x & 1) == 0) atomicMax(s_amax + h * kP + p, __float_as_uint(m));
}

// ---- steps from the absolute maxima
__global__ void calib_steps_kernel(const uint32_t* __restrict__ xs_amax,
                                   const uint32_t* __restrict__ s_amax,
                                   const uint32_t* __restrict__ cb_amax, float* __restrict__ aXs,
                                   float* __restrict__ aS, float* __restrict__ aCB, int H, int G,
                                   int xs_per_head) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t < H * kP) {
    const float sm = __uint_as_float(s_amax[t]);
    const float a = (float)((double)sm / 127.0);
    aS[t] = a == 0.0f ? 1.0f : a;
    if (!xs_per_head) {
      const float x = __uint_as_float(xs_amax[t]) / 127.0f;
      aXs[t] = x == 0.0f ? 1.0f : x;
    }
  }
  if (xs_per_head && t < H) {
    float m = 0.0f;
    for (int p = 0; p < kP; ++p) m = __builtin_fmaxf(m, __uint_as_float(xs_amax[t * kP + p]));
    const float x = m / 127.0f;
    aXs[t] = x == 0.0f ? 1.0f : x;
  }
  if (t < G) {
    const float a = (float)((double)__uint_as_float(cb_amax[t]) / 127.0);
    aCB[t] = a == 0.0f ? 1.0f : a;
  }
}

// ---- corr[h, p] = eta * mean over (b, l) of (y_fp - y_q), in fp64 and in a fixed order: stage 1
//      sums token block nb of head h (blockIdx = (h, nb)) per channel, stage 2 adds the blocks
constexpr int kCorrBlocks = 64;

__global__ __launch_bounds__(256) void calib_corr_partial(const float* __restrict__ y_fp,
                                                          const float* __restrict__ y_q,
                                                          double* __restrict__ part, int64_t T,
                                                          int H) {
  __shared__ double s_sum[4][kP];
  const int t = threadIdx.x, p = t & 63, q = t >> 6;
  const int h = blockIdx.x, nb = blockIdx.y, nbs = gridDim.y;
  const int64_t t0 = T * nb / nbs, t1 = T * (nb + 1) / nbs;
  const size_t HP = (size_t)H * kP;
  double sum = 0.0;
  for (int64_t tok = t0 + q; tok < t1; tok += 4) {
    const size_t i = (size_t)tok * HP + (size_t)h * kP + p;
    sum += (double)y_fp[i] - (double)y_q[i];
  }
  s_sum[q][p] = sum;
  __syncthreads();
  if (t < kP)
    part[((size_t)h * nbs + nb) * kP + t] = s_sum[0][t] + s_sum[1][t] + s_sum[2][t] + s_sum[3][t];
}

__global__ void calib_corr_final(const double* __restrict__ part, float* __restrict__ corr,
                                 int64_t T, int H, int nbs, float eta) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= H * kP) return;
  const int h = i / kP, p = i - h * kP;
  double s = 0.0;
  for (int nb = 0; nb < nbs; ++nb) s += part[((size_t)h * nbs + nb) * kP + p];
  corr[i] = (float)((double)eta * s / (double)T);
}

__global__ void zero_u32(uint32_t* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

}  // namespace

hipError_t launch_calib_zero(uint32_t* p, int n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_u32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

hipError_t launch_calib_xs(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                           int dt_softplus, const float* A, uint32_t* xs_amax, hipStream_t st) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.nheads;
  if (nwork == 0) return hipSuccess;
  if (x_dtype == 1)
    hipLaunchKernelGGL(calib_xs_kernel<_Float16>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const _Float16*>(x), dt, A, dt_softplus, xs_amax, d.seqlen,
                       d.nheads, d.nchunks);
  else
    hipLaunchKernelGGL(calib_xs_kernel<float>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const float*>(x), dt, A, dt_softplus, xs_amax, d.seqlen,
                       d.nheads, d.nchunks);
  return hipGetLastError();
}

hipError_t launch_calib_states(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                               int dt_softplus, const float* A, const _Float16* bT_frag,
                               float* S, double* dec64, uint32_t* s_amax, hipStream_t st) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.nheads;
  if (nwork == 0) return hipSuccess;
  if (x_dtype == 1)
    hipLaunchKernelGGL(calib_state_kernel<_Float16>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const _Float16*>(x), dt, A, bT_frag, dt_softplus, S, dec64,
                       d.seqlen, d.nheads, d.ngroups, d.nchunks);
  else
    hipLaunchKernelGGL(calib_state_kernel<float>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const float*>(x), dt, A, bT_frag, dt_softplus, S, dec64,
                       d.seqlen, d.nheads, d.ngroups, d.nchunks);
  const int64_t nthreads = (int64_t)d.batch * d.nheads * kP * kN / 4;
  hipLaunchKernelGGL(calib_pass_kernel, dim3((unsigned)((nthreads + 255) / 256)), dim3(256), 0,
                     st, S, dec64, s_amax, d.nchunks, d.nheads, nthreads);
  return hipGetLastError();
}

hipError_t launch_calib_steps(const uint32_t* xs_amax, const uint32_t* s_amax,
                              const uint32_t* cb_amax, float* aXs, float* aS, float* aCB, int H,
                              int G, int xs_per_head, hipStream_t st) {
  const int n = H * kP > G ? H * kP : G;
  hipLaunchKernelGGL(calib_steps_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     xs_amax, s_amax, cb_amax, aXs, aS, aCB, H, G, xs_per_head);
  return hipGetLastError();
}

size_t calib_corr_scratch_bytes(int H) { return (size_t)H * kCorrBlocks * kP * sizeof(double); }

hipError_t launch_calib_corr(const float* y_fp, const float* y_q, double* part, float* corr,
                             int64_t T, int H, float eta, hipStream_t st) {
  const int64_t nb = T / 256 < 1 ? 1 : (T / 256 > kCorrBlocks ? kCorrBlocks : T / 256);
  hipLaunchKernelGGL(calib_corr_partial, dim3((unsigned)H, (unsigned)nb), dim3(256), 0, st, y_fp,
                     y_q, part, T, H);
  hipLaunchKernelGGL(calib_corr_final, dim3((unsigned)((H * kP + 255) / 256)), dim3(256), 0, st,
                     part, corr, T, H, (int)nb, eta);
  return hipGetLastError();
}

}  // namespace ssdi8
