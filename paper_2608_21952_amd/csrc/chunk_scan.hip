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
// once per chunk in fp64 and rounded to fp32, so an off-diagonal weight costs two fp32 products
// and no exp; only the 8 diagonal blocks evaluate exp per element.
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
constexpr int kBuf = (kP * kXTS > kQ * kYS) ? kP * kXTS : kQ * kYS;

template <typename XT>
__device__ __forceinline__ void load_pair_h(const XT* p, _Float16& a, _Float16& b);

template <>
__device__ __forceinline__ void load_pair_h<_Float16>(const _Float16* p, _Float16& a,
                                                      _Float16& b) {
  const uint32_t v = *reinterpret_cast<const uint32_t*>(p);
  a = __builtin_bit_cast(_Float16, (uint16_t)(v & 0xffffu));
  b = __builtin_bit_cast(_Float16, (uint16_t)(v >> 16));
}

template <>
__device__ __forceinline__ void load_pair_h<float>(const float* p, _Float16& a, _Float16& b) {
  const float2 v = *reinterpret_cast<const float2*>(p);
  a = (_Float16)v.x;
  b = (_Float16)v.y;
}

__device__ __forceinline__ uint32_t pack2_h(_Float16 a, _Float16 b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

template <typename XT, typename YT>
__global__ __launch_bounds__(256) void chunk_scan_kernel(
    const XT* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const int8_t* __restrict__ Cq, const float* __restrict__ C_scale, int c_per_token,
    const int8_t* __restrict__ pin, const int8_t* __restrict__ cbq,
    const float* __restrict__ cb_scale, const float* __restrict__ state_scale,
    const float* __restrict__ Dv, const float* __restrict__ corr, int dt_softplus,
    YT* __restrict__ y, int32_t* __restrict__ y1_tap, int L, int H, int G, int nc) {
  __shared__ __attribute__((aligned(16))) uint8_t s_buf[kBuf];
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

  // ---- ChunkCumsum (recomputed: exact fp64 sums give the same cs as the ChunkState kernel)
  float dtv = dt[(tok0 + t) * H + h];
  if (dt_softplus) dtv = softplus_f32(dtv);
  const float dA = dtv * A[h];
  const double cs = block_scan_f64_256((double)dA, s_scan);
  s_cs[t] = cs;
  __syncthreads();
  {
    const int blk = t >> 5;
    const float dtcb = aCB * dtv;
    s_dtcb[t] = dtcb;
    s_u[t] = (float)((double)dtcb * exp(s_cs[blk * 32 + 31] - cs));
    s_vp[t] = blk ? (float)exp(cs - s_cs[blk * 32 - 1]) : 1.0f;
    const float ac = c_per_token ? C_scale[(tok0 + t) * G + g] : C_scale[g];
    s_eoff[t] = (float)((double)ac * exp(cs));
    if (t < 64) {
      const int ra = t >> 3, rb = t & 7;
      s_R[ra][rb] = (rb <= ra) ? (float)exp(s_cs[ra * 32 + 31] - s_cs[rb * 32 + 31]) : 0.0f;
    }
  }
  // ---- stage x^T [p][i] as fp16.  Thread: channel pair (p0, p0+1), tokens [32 jb, 32 jb + 32)
  {
    const int pp = t & 31, jb = t >> 5, p0 = 2 * pp;
    uint32_t w0[16], w1[16];
#pragma unroll
    for (int r2 = 0; r2 < 16; ++r2) {
      _Float16 a0, b0, a1, b1;
      const int j = jb * 32 + 2 * r2;
      load_pair_h<XT>(x + (tok0 + j) * HP + (size_t)h * kP + p0, a0, b0);
      load_pair_h<XT>(x + (tok0 + j + 1) * HP + (size_t)h * kP + p0, a1, b1);
      w0[r2] = pack2_h(a0, a1);
      w1[r2] = pack2_h(b0, b1);
    }
    uint8_t* r0 = s_buf + p0 * kXTS + jb * 64;
    uint8_t* r1 = r0 + kXTS;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *reinterpret_cast<uint4*>(r0 + 16 * q) =
          make_uint4(w0[4 * q], w0[4 * q + 1], w0[4 * q + 2], w0[4 * q + 3]);
      *reinterpret_cast<uint4*>(r1 + 16 * q) =
          make_uint4(w1[4 * q], w1[4 * q + 1], w1[4 * q + 2], w1[4 * q + 3]);
    }
  }
  __syncthreads();

  const int8_t* pbase = pin + (((size_t)b * nc + c) * H + h) * (size_t)kP * kN;
  const int8_t* cbbase = cbq + (((size_t)b * nc + c) * G + g) * (size_t)kQ * kQ;
  const float aS0 = state_scale[h * kP + (lane & 31)];
  const float aS1 = state_scale[h * kP + 32 + (lane & 31)];
  const float cr0 = corr ? corr[h * kP + (lane & 31)] : 0.0f;
  const float cr1 = corr ? corr[h * kP + 32 + (lane & 31)] : 0.0f;
  const float Dh = Dv ? Dv[h] : 0.0f;

  uint32_t outh[2][2][8];  // packed fp16 results [j-block][p-tile][register pair]

#pragma unroll
  for (int q2 = 0; q2 < 2; ++q2) {
    const int jt = q2 ? 7 - wv : wv;
    const int jrow = jt * 32 + (lane & 31);
    // -- Scan1: int8 MFMA over n
    v16i yi0 = {}, yi1 = {};
    {
      const int8_t* crow = Cq + ((tok0 + jrow) * G + g) * kN;
      const int8_t* p0row = pbase + (size_t)(lane & 31) * kN;
      const int8_t* p1row = p0row + 32 * kN;
#pragma unroll
      for (int ks = 0; ks < kN / 32; ++ks) {
        const int kof = ks * 32 + 16 * (lane >> 5);
        const v4i a = *reinterpret_cast<const v4i*>(crow + kof);
        const v4i b0 = *reinterpret_cast<const v4i*>(p0row + kof);
        const v4i b1 = *reinterpret_cast<const v4i*>(p1row + kof);
        yi0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b0, yi0, 0, 0, 0);
        yi1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b1, yi1, 0, 0, 0);
      }
    }
    // -- Scan2: fp16 MFMA over the causal source tokens i
    v16f yd0 = {}, yd1 = {};
    {
      const int8_t* cbrow = cbbase + (size_t)jrow * kQ;
      const double csj = s_cs[jrow];
      const float vpj = s_vp[jrow];
      for (int it = 0; it <= jt; ++it) {
        const float vj = (it < jt) ? vpj * s_R[jt - 1][it] : 0.0f;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int i0 = it * 32 + ks * 16 + 8 * (lane >> 5);
          const uint2 cb8 = *reinterpret_cast<const uint2*>(cbrow + i0);
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
          const v8h b0 = *reinterpret_cast<const v8h*>(s_buf + (lane & 31) * kXTS + i0 * 2);
          const v8h b1 =
              *reinterpret_cast<const v8h*>(s_buf + (32 + (lane & 31)) * kXTS + i0 * 2);
          yd0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(wf, b0, yd0, 0, 0, 0);
          yd1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(wf, b1, yd1, 0, 0, 0);
        }
      }
    }
    // -- epilogue for this j-block
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = jt * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      const float eo = s_eoff[j];
      const size_t orow = (tok0 + j) * HP + (size_t)h * kP;
      float x0, x1;
      if constexpr (sizeof(XT) == 2) {
        x0 = (float)*reinterpret_cast<const _Float16*>(s_buf + (lane & 31) * kXTS + j * 2);
        x1 = (float)*reinterpret_cast<const _Float16*>(s_buf + (32 + (lane & 31)) * kXTS +
                                                       j * 2);
      } else {
        x0 = (float)x[orow + (lane & 31)];
        x1 = (float)x[orow + 32 + (lane & 31)];
      }
      const float v0 = ((float)yi0[r] * eo) * aS0 + yd0[r] + Dh * x0 + cr0;
      const float v1 = ((float)yi1[r] * eo) * aS1 + yd1[r] + Dh * x1 + cr1;
      if (y1_tap) {
        y1_tap[orow + (lane & 31)] = yi0[r];
        y1_tap[orow + 32 + (lane & 31)] = yi1[r];
      }
      if constexpr (sizeof(YT) == 4) {
        y[orow + (lane & 31)] = v0;
        y[orow + 32 + (lane & 31)] = v1;
      } else {
        const _Float16 h0 = (_Float16)v0, h1 = (_Float16)v1;
        if (r & 1) {
          outh[q2][0][r >> 1] |= (uint32_t)__builtin_bit_cast(uint16_t, h0) << 16;
          outh[q2][1][r >> 1] |= (uint32_t)__builtin_bit_cast(uint16_t, h1) << 16;
        } else {
          outh[q2][0][r >> 1] = (uint32_t)__builtin_bit_cast(uint16_t, h0);
          outh[q2][1][r >> 1] = (uint32_t)__builtin_bit_cast(uint16_t, h1);
        }
      }
    }
  }

  if constexpr (sizeof(YT) == 2) {
    __syncthreads();  // x^T no longer read: reuse the buffer as the output stage [j][p]
#pragma unroll
    for (int q2 = 0; q2 < 2; ++q2) {
      const int jt = q2 ? 7 - wv : wv;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int j = jt * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const uint32_t sh = (r & 1) ? 16 : 0;
        *reinterpret_cast<uint16_t*>(s_buf + j * kYS + (lane & 31) * 2) =
            (uint16_t)(outh[q2][0][r >> 1] >> sh);
        *reinterpret_cast<uint16_t*>(s_buf + j * kYS + (32 + (lane & 31)) * 2) =
            (uint16_t)(outh[q2][1][r >> 1] >> sh);
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < (kQ * kP * 2) / (16 * 256); ++k) {
      const int idx = k * 256 + t;
      const int j = idx >> 3, col = idx & 7;
      *reinterpret_cast<uint4*>(reinterpret_cast<uint8_t*>(y) +
                                ((tok0 + j) * HP + (size_t)h * kP) * 2 + col * 16) =
          *reinterpret_cast<const uint4*>(s_buf + j * kYS + col * 16);
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
