// FP16 baseline, ChunkCumsum + ChunkState and StatePassing (Alg. 2 modules 1-3 without
// quantization):
//   dt, dA, cs, LUT_state    as in the INT8 ChunkState (fp64 softplus and in-chunk sum)
//   X~       = fp16(fl32(LUT_j x_jp))
//   S[p, n]  = sum_j X~[j, p] B[j, n]       fp16 MFMA 32x32x16 over tokens, fp32 accumulation
//   d        = fl32(exp(cs_last))
//   P_in[c+1] = fl32(d P_in[c] + S[c])      one fma per element, fp32 states
// S and P_in are kept in the fragment order of ChunkScan1's fp16 operand (frag::k16_offset with
// rows p, K = n, fp32 elements); the initial and final states are row-major [p][n].
#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kXS = kQ * 2 + 16;   // LDS bytes per channel row of X~^T (fp16)

typedef _Float16 h8 __attribute__((ext_vector_type(8)));

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

template <typename XT>
__global__ __launch_bounds__(256) void fp16_state_kernel(
    const XT* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const _Float16* __restrict__ bT_frag, int dt_softplus, float* __restrict__ S,
    float* __restrict__ dec, int L, int H, int G, int nc) {
  __shared__ __attribute__((aligned(16))) uint8_t s_x[kP * kXS];
  __shared__ float s_lut[kQ];
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

  const int pp = t & 31, jb = t >> 5, p0 = 2 * pp;
  typename Pair<XT>::raw xr[32];
  {
    const XT* xb = x + (tok0 + (size_t)jb * 32) * HP + (size_t)h * kP + p0;
#pragma unroll
    for (int r = 0; r < 32; ++r) xr[r] = Pair<XT>::load(xb + (size_t)r * HP);
  }

  float dtv = dt[(tok0 + t) * H + h];
  if (dt_softplus) dtv = softplus_f32(dtv);
  const float dA = dtv * A[h];
  const double cs = block_scan_f64_256(dA, s_scan, s_lut);
  if (t == kQ - 1) s_last = cs;
  __syncthreads();
  const double last = s_last;
  s_lut[t] = dtv * (float)exp(last - cs);
  if (t == 0) dec[((size_t)b * H + h) * nc + c] = (float)exp(last);
  __syncthreads();

  // ---- X~ = fp16(LUT x), written transposed to LDS ([p][j], tokens contiguous)
  {
    uint32_t w0[16], w1[16];
#pragma unroll
    for (int r2 = 0; r2 < 16; ++r2) {
      const int r = 2 * r2;
      const float l0 = s_lut[jb * 32 + r], l1 = s_lut[jb * 32 + r + 1];
      const _Float16 a0 = (_Float16)(l0 * Pair<XT>::lo(xr[r]));
      const _Float16 a1 = (_Float16)(l1 * Pair<XT>::lo(xr[r + 1]));
      const _Float16 c0 = (_Float16)(l0 * Pair<XT>::hi(xr[r]));
      const _Float16 c1 = (_Float16)(l1 * Pair<XT>::hi(xr[r + 1]));
      w0[r2] = (uint32_t)__builtin_bit_cast(uint16_t, a0) |
               ((uint32_t)__builtin_bit_cast(uint16_t, a1) << 16);
      w1[r2] = (uint32_t)__builtin_bit_cast(uint16_t, c0) |
               ((uint32_t)__builtin_bit_cast(uint16_t, c1) << 16);
    }
    uint8_t* r0 = s_x + p0 * kXS + jb * 64;
    uint8_t* r1 = r0 + kXS;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *reinterpret_cast<uint4*>(r0 + 16 * q) =
          make_uint4(w0[4 * q], w0[4 * q + 1], w0[4 * q + 2], w0[4 * q + 3]);
      *reinterpret_cast<uint4*>(r1 + 16 * q) =
          make_uint4(w1[4 * q], w1[4 * q + 1], w1[4 * q + 2], w1[4 * q + 3]);
    }
  }
  __syncthreads();

  // ---- S = X~^T B: wave -> p-tile mt (32 rows), n-tiles ntb, ntb + 1
  const int mt = wv & 1, ntb = (wv >> 1) * 2, half = lane >> 5;
  const _Float16* bq = bT_frag + (((size_t)b * nc + c) * G + g) * (size_t)kN * kQ;
  v16f acc0 = {}, acc1 = {};
  {
    const uint8_t* arow = s_x + (mt * 32 + (lane & 31)) * kXS + 16 * half;
    const _Float16* b0f = bq + (size_t)ntb * (kQ / 16) * 512 + lane * 8;
    const _Float16* b1f = b0f + (size_t)(kQ / 16) * 512;
#pragma unroll
    for (int ks = 0; ks < kQ / 16; ++ks) {
      const h8 a = *reinterpret_cast<const h8*>(arow + ks * 32);
      const h8 b0 = *reinterpret_cast<const h8*>(b0f + ks * 512);
      const h8 b1 = *reinterpret_cast<const h8*>(b1f + ks * 512);
      acc0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b1, acc1, 0, 0, 0);
    }
  }
  __syncthreads();   // X~^T no longer read: its LDS stages S

  // ---- stage S in ChunkScan1 fragment order (fp32), then 16-byte copies out
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

// P_in[c+1] = fl32(d[c] P_in[c] + S[c]) over [b, c, h, P*N] fp32 in fragment order, 4 elements
// per thread, two batches of 8 chunks of loads in flight.
__global__ __launch_bounds__(256) void fp16_pass_kernel(
    const float* __restrict__ S, const float* __restrict__ dec, const float* __restrict__ init,
    float* __restrict__ pin, float* __restrict__ final_state, int nc, int H, int64_t nthreads) {
  constexpr int kDepth = 8;
  constexpr int64_t kE = (int64_t)kP * kN;
  const int64_t gt = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (gt >= nthreads) return;
  const int64_t e = gt * 4;
  const int64_t bh = e / kE;
  const int64_t off = e - bh * kE;
  const int64_t b = bh / H, h = bh - b * H;
  int row, k;
  frag::k16_coords((size_t)off, kN, &row, &k);
  const int64_t roff = (int64_t)row * kN + k;   // row-major offset of the same 4 elements
  float4 st = init ? *reinterpret_cast<const float4*>(init + bh * kE + roff)
                   : make_float4(0.f, 0.f, 0.f, 0.f);
  const size_t cstride = (size_t)H * kE;
  const size_t base = ((size_t)b * nc * H + h) * kE + off;
  const float* drow = dec + bh * nc;
  for (int c0 = 0; c0 < nc; c0 += kDepth) {
    float4 v[kDepth];
    float d[kDepth];
#pragma unroll
    for (int q = 0; q < kDepth; ++q) {
      if (c0 + q < nc) {
        v[q] = *reinterpret_cast<const float4*>(S + base + (size_t)(c0 + q) * cstride);
        d[q] = drow[c0 + q];
      }
    }
#pragma unroll
    for (int q = 0; q < kDepth; ++q) {
      if (c0 + q < nc) {
        *reinterpret_cast<float4*>(pin + base + (size_t)(c0 + q) * cstride) = st;
        st.x = __builtin_fmaf(d[q], st.x, v[q].x);
        st.y = __builtin_fmaf(d[q], st.y, v[q].y);
        st.z = __builtin_fmaf(d[q], st.z, v[q].z);
        st.w = __builtin_fmaf(d[q], st.w, v[q].w);
      }
    }
  }
  if (final_state) *reinterpret_cast<float4*>(final_state + bh * kE + roff) = st;
}

}  // namespace

hipError_t launch_fp16_state(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                             int dt_softplus, const float* A, const _Float16* bT_frag, float* S,
                             float* dec, hipStream_t st) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.nheads;
  if (nwork == 0) return hipSuccess;
  if (x_dtype == 1)
    hipLaunchKernelGGL(fp16_state_kernel<_Float16>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const _Float16*>(x), dt, A, bT_frag, dt_softplus, S, dec,
                       d.seqlen, d.nheads, d.ngroups, d.nchunks);
  else
    hipLaunchKernelGGL(fp16_state_kernel<float>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const float*>(x), dt, A, bT_frag, dt_softplus, S, dec,
                       d.seqlen, d.nheads, d.ngroups, d.nchunks);
  return hipGetLastError();
}

hipError_t launch_fp16_pass(const LayerDims& d, const float* S, const float* dec,
                            const float* init, float* pin, float* final_state, hipStream_t st) {
  const int64_t nthreads = (int64_t)d.batch * d.nheads * kP * kN / 4;
  if (nthreads == 0) return hipSuccess;
  hipLaunchKernelGGL(fp16_pass_kernel, dim3((unsigned)((nthreads + 255) / 256)), dim3(256), 0,
                     st, S, dec, init, pin, final_state, d.nchunks, d.nheads, nthreads);
  return hipGetLastError();
}

}  // namespace ssdi8
