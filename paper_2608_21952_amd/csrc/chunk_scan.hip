// ChunkScan1 (INT8) + ChunkScan2 (FP16) + output epilogue (Alg. 2 modules 5-6, Sec. 4.2, Eq. 10).
//
// One workgroup per (batch, chunk, head); output tile y[256 tokens j][64 channels p].
//   Scan1  Y1[j,p] = sum_n C_q[j,n] P_in[p,n]        int8 MFMA (K = n, both operands n-major)
//          y_off   = Y1 * (a_C exp(cs_j)) * a_S[p]   decay and dequant applied after the product
//   Scan2  W[j,i]  = fp16(CB_q[j,i] * a_CB * dt_i * exp(cs_j - cs_i)),  i <= j
//          y_diag  = W . fp16(x)                    fp16 MFMA, fp32 accumulation (K = tokens i)
//   y = y_off + y_diag + D[h] x + corr[h,p]  -> fp16 / fp32
//
// The segment-sum decay exp(cs_j - cs_i) is decoupled from the Q x Q weight construction on the
// off-diagonal 32x32 blocks: with r_t = cs at the last token of block t,
//   exp(cs_j - cs_i) = exp(cs_j - r_{J-1}) * exp(r_{J-1} - r_I) * exp(r_I - cs_i)
// (J, I the blocks of j, i; every factor <= 1, so nothing overflows and an underflow only
// happens where the true weight underflows).  The row / block / column factors are computed
// once per chunk (fp32 exp of differences formed from the fp64 sums), so an off-diagonal weight
// costs two fp32 products and no exp; only the 8 diagonal blocks evaluate exp per element.
//
// Work split: wave w owns the j-blocks {w, 7-w} (1+w + 8-w = 9 causal block pairs per wave).
// x is staged once in LDS as x^T [p][i] (fp16, tokens contiguous = the Scan2 MFMA K-slice) and
// also serves the D skip term; the fp16 output leaves through an LDS stage as 128-byte rows.
#include "common.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kXTS = kQ * 2 + 16;   // bytes per channel row of x^T (fp16)
constexpr int kYS = kP * 2 + 16;    // bytes per token row of the staged fp16 output

// Two adjacent channels of one token row, loaded raw and converted to fp16 for the MFMA.
template <typename XT> struct Pair;
template <> struct Pair<_Float16> {
  typedef uint32_t raw;
  static __device__ __forceinline__ raw load(const _Float16* p) {
    return *reinterpret_cast<const uint32_t*>(p);
  }
  static __device__ __forceinline__ uint16_t lo(raw v) { return (uint16_t)(v & 0xffffu); }
  static __device__ __forceinline__ uint16_t hi(raw v) { return (uint16_t)(v >> 16); }
};
template <> struct Pair<float> {
  typedef float2 raw;
  static __device__ __forceinline__ raw load(const float* p) {
    return *reinterpret_cast<const float2*>(p);
  }
  static __device__ __forceinline__ uint16_t lo(raw v) {
    return __builtin_bit_cast(uint16_t, (_Float16)v.x);
  }
  static __device__ __forceinline__ uint16_t hi(raw v) {
    return __builtin_bit_cast(uint16_t, (_Float16)v.y);
  }
};

// fp32 softplus (the output path only needs dt to fp32 accuracy).
__device__ __forceinline__ float softplus_fast(float v) {
  return v > 20.0f ? v : log1pf(expf(v));
}

template <typename XT, typename YT>
__global__ __launch_bounds__(256, 2) void chunk_scan_kernel(
    const XT* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const int8_t* __restrict__ Cq, const float* __restrict__ C_scale, int c_per_token,
    const int8_t* __restrict__ pin, const int8_t* __restrict__ cbq,
    const float* __restrict__ cb_scale, const float* __restrict__ state_scale,
    const float* __restrict__ Dv, const float* __restrict__ corr, int dt_softplus,
    YT* __restrict__ y, int32_t* __restrict__ y1_tap, int L, int H, int G, int nc) {
  __shared__ __attribute__((aligned(16))) uint8_t s_xT[kP * kXTS];
  __shared__ __attribute__((aligned(16))) uint8_t s_y[sizeof(YT) == 2 ? kQ * kYS : 16];
  __shared__ double s_cs[kQ];
  __shared__ float s_u[kQ];     // a_CB dt_i exp(r_I - cs_i)
  __shared__ float s_dtcb[kQ];  // a_CB dt_i
  __shared__ float s_vp[kQ];    // exp(cs_j - r_{J-1})
  __shared__ float s_eoff[kQ];  // a_C(j) exp(cs_j)
  __shared__ float s_R[8][8];   // exp(r_a - r_b), b <= a
  __shared__ double s_scan[4];

  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int h = w % H;
  const int bc = w / H;
  const int c = bc % nc;
  const int b = bc / nc;
  const int g = h / (H / G);
  const size_t tok0 = (size_t)b * L + (size_t)c * kQ;
  const size_t HP = (size_t)H * kP;
  const float aCB = cb_scale[g];

  // ---- x tile loads first (thread: channel pair (p0, p0+1), tokens [32 jb, 32 jb + 32))
  const int pp = t & 31, jb = t >> 5, p0 = 2 * pp;
  typename Pair<XT>::raw xr[32];
  {
    const XT* xb = x + (tok0 + (size_t)jb * 32) * HP + (size_t)h * kP + p0;
#pragma unroll
    for (int r = 0; r < 32; ++r) xr[r] = Pair<XT>::load(xb + (size_t)r * HP);
  }

  // ---- ChunkCumsum (fp64 sums; the factors derived from it only need fp32 accuracy here)
  float dtv = dt[(tok0 + t) * H + h];
  if (dt_softplus) dtv = softplus_fast(dtv);
  const float dA = dtv * A[h];
  const double cs = block_scan_f64_256((double)dA, s_scan);
  s_cs[t] = cs;
  __syncthreads();
  {
    const int blk = t >> 5;
    const float dtcb = aCB * dtv;
    s_dtcb[t] = dtcb;
    s_u[t] = dtcb * expf((float)(s_cs[blk * 32 + 31] - cs));
    s_vp[t] = blk ? expf((float)(cs - s_cs[blk * 32 - 1])) : 1.0f;
    const float ac = c_per_token ? C_scale[(tok0 + t) * G + g] : C_scale[g];
    s_eoff[t] = ac * expf((float)cs);
    if (t < 64) {
      const int ra = t >> 3, rb = t & 7;
      s_R[ra][rb] = (rb <= ra) ? expf((float)(s_cs[ra * 32 + 31] - s_cs[rb * 32 + 31])) : 0.0f;
    }
  }
  // ---- x^T [p][i] as fp16 in LDS (tokens contiguous = the ChunkScan2 MFMA K-slice)
  {
    uint8_t* r0 = s_xT + p0 * kXTS + jb * 64;
    uint8_t* r1 = r0 + kXTS;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t a[4], bb[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = 8 * q + 2 * u;
        a[u] = (uint32_t)Pair<XT>::lo(xr[r]) | ((uint32_t)Pair<XT>::lo(xr[r + 1]) << 16);
        bb[u] = (uint32_t)Pair<XT>::hi(xr[r]) | ((uint32_t)Pair<XT>::hi(xr[r + 1]) << 16);
      }
      *reinterpret_cast<uint4*>(r0 + 16 * q) = make_uint4(a[0], a[1], a[2], a[3]);
      *reinterpret_cast<uint4*>(r1 + 16 * q) = make_uint4(bb[0], bb[1], bb[2], bb[3]);
    }
  }
  __syncthreads();

  const int8_t* pbase = pin + (((size_t)b * nc + c) * H + h) * (size_t)kP * kN;
  const int8_t* cbbase = cbq + (((size_t)b * nc + c) * G + g) * (size_t)kQ * kQ;
  const int pc = lane & 31, half = lane >> 5;
  const float aS0 = state_scale[h * kP + pc];
  const float aS1 = state_scale[h * kP + 32 + pc];
  const float cr0 = corr ? corr[h * kP + pc] : 0.0f;
  const float cr1 = corr ? corr[h * kP + 32 + pc] : 0.0f;
  const float Dh = Dv ? Dv[h] : 0.0f;

  for (int q2 = 0; q2 < 2; ++q2) {
    const int jt = q2 ? 7 - wv : wv;
    const int jrow = jt * 32 + pc;
    // -- Scan1: int8 MFMA over n (C_q rows against the entering state rows)
    v16i yi0 = {}, yi1 = {};
    {
      const int8_t* crow = Cq + ((tok0 + jrow) * G + g) * kN + 16 * half;
      const int8_t* p0row = pbase + (size_t)pc * kN + 16 * half;
      const int8_t* p1row = p0row + 32 * kN;
      v4i a[4], b0[4], b1[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        a[ks] = *reinterpret_cast<const v4i*>(crow + 32 * ks);
        b0[ks] = *reinterpret_cast<const v4i*>(p0row + 32 * ks);
        b1[ks] = *reinterpret_cast<const v4i*>(p1row + 32 * ks);
      }
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        yi0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[ks], b0[ks], yi0, 0, 0, 0);
        yi1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[ks], b1[ks], yi1, 0, 0, 0);
      }
    }
    // -- Scan2: fp16 MFMA over the causal source tokens i, CB_q of block it+1 prefetched
    v16f yd0 = {}, yd1 = {};
    {
      const int8_t* cbrow = cbbase + (size_t)jrow * kQ + 8 * half;
      const double csj = s_cs[jrow];
      const float vpj = s_vp[jrow];
      uint2 cur0 = *reinterpret_cast<const uint2*>(cbrow);
      uint2 cur1 = *reinterpret_cast<const uint2*>(cbrow + 16);
      for (int it = 0; it <= jt; ++it) {
        uint2 nx0 = cur0, nx1 = cur1;
        if (it < jt) {
          nx0 = *reinterpret_cast<const uint2*>(cbrow + (it + 1) * 32);
          nx1 = *reinterpret_cast<const uint2*>(cbrow + (it + 1) * 32 + 16);
        }
        const float vj = (it < jt) ? vpj * s_R[jt - 1][it] : 0.0f;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const uint2 cb8 = ks ? cur1 : cur0;
          const int i0 = it * 32 + ks * 16 + 8 * half;
          v8h wf;
          if (it < jt) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int cbv = sext8(e < 4 ? cb8.x : cb8.y, e & 3);
              wf[e] = (_Float16)(((float)cbv * s_u[i0 + e]) * vj);
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int i = i0 + e;
              const int cbv = sext8(e < 4 ? cb8.x : cb8.y, e & 3);
              float wv_ = 0.0f;
              if (i <= jrow) wv_ = ((float)cbv * s_dtcb[i]) * __expf((float)(csj - s_cs[i]));
              wf[e] = (_Float16)wv_;
            }
          }
          const v8h xb0 = *reinterpret_cast<const v8h*>(s_xT + pc * kXTS + i0 * 2);
          const v8h xb1 = *reinterpret_cast<const v8h*>(s_xT + (32 + pc) * kXTS + i0 * 2);
          yd0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(wf, xb0, yd0, 0, 0, 0);
          yd1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(wf, xb1, yd1, 0, 0, 0);
        }
        cur0 = nx0;
        cur1 = nx1;
      }
    }
    // -- epilogue for this j-block: y = y_off + y_diag + D x + corr
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = jt * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
      const float eo = s_eoff[j];
      const size_t orow = (tok0 + j) * HP + (size_t)h * kP;
      float x0, x1;
      if constexpr (sizeof(XT) == 2) {
        x0 = (float)*reinterpret_cast<const _Float16*>(s_xT + pc * kXTS + j * 2);
        x1 = (float)*reinterpret_cast<const _Float16*>(s_xT + (32 + pc) * kXTS + j * 2);
      } else {
        x0 = (float)x[orow + pc];
        x1 = (float)x[orow + 32 + pc];
      }
      const float v0 = ((float)yi0[r] * eo) * aS0 + yd0[r] + Dh * x0 + cr0;
      const float v1 = ((float)yi1[r] * eo) * aS1 + yd1[r] + Dh * x1 + cr1;
      if (y1_tap) {
        y1_tap[orow + pc] = yi0[r];
        y1_tap[orow + 32 + pc] = yi1[r];
      }
      if constexpr (sizeof(YT) == 4) {
        y[orow + pc] = v0;
        y[orow + 32 + pc] = v1;
      } else {
        *reinterpret_cast<_Float16*>(s_y + j * kYS + pc * 2) = (_Float16)v0;
        *reinterpret_cast<_Float16*>(s_y + j * kYS + (32 + pc) * 2) = (_Float16)v1;
      }
    }
  }

  if constexpr (sizeof(YT) == 2) {
    __syncthreads();
#pragma unroll
    for (int k = 0; k < (kQ * kP * 2) / (16 * 256); ++k) {
      const int idx = k * 256 + t;
      const int j = idx >> 3, col = idx & 7;
      *reinterpret_cast<uint4*>(reinterpret_cast<uint8_t*>(y) +
                                ((tok0 + j) * HP + (size_t)h * kP) * 2 + col * 16) =
          *reinterpret_cast<const uint4*>(s_y + j * kYS + col * 16);
    }
  }
}

}  // namespace

hipError_t launch_chunk_scan(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                             int dt_softplus, const float* A, const int8_t* Cq,
                             const float* C_scale, int c_per_token, const int8_t* pin,
                             const int8_t* cbq, const float* cb_scale, const float* state_scale,
                             const float* D, const float* corr, void* y, int y_dtype,
                             int32_t* y1_tap, hipStream_t st) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.nheads;
  if (nwork == 0) return hipSuccess;
  const dim3 grid((unsigned)nwork), block(256);
#define SSDI8_SCAN_LAUNCH(XT, YT)                                                             \
  hipLaunchKernelGGL((chunk_scan_kernel<XT, YT>), grid, block, 0, st,                         \
                     static_cast<const XT*>(x), dt, A, Cq, C_scale, c_per_token, pin, cbq,    \
                     cb_scale, state_scale, D, corr, dt_softplus, static_cast<YT*>(y), y1_tap, \
                     d.seqlen, d.nheads, d.ngroups, d.nchunks)
  if (x_dtype == 1 && y_dtype == 1) SSDI8_SCAN_LAUNCH(_Float16, _Float16);
  else if (x_dtype == 1) SSDI8_SCAN_LAUNCH(_Float16, float);
  else if (y_dtype == 1) SSDI8_SCAN_LAUNCH(float, _Float16);
  else SSDI8_SCAN_LAUNCH(float, float);
#undef SSDI8_SCAN_LAUNCH
  return hipGetLastError();
}

}  // namespace ssdi8
