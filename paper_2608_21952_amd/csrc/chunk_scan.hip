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
// in row order [j][p] for the D skip term; the fp16 output is written over the x rows and leaves
// through that stage as 128-byte rows.
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
  constexpr bool kHalfX = sizeof(XT) == 2;
  // One LDS block with the small per-token tables first, so that their offsets fit the 16-bit
  // ds offset field (separate __shared__ arrays may be placed large-first).
  struct __attribute__((aligned(16))) Smem {
    // Column tables of the ChunkScan2 weights, interleaved as (w, -128 w) pairs so that an int8
    // weight q, converted as the unsigned byte q + 128, gives fl32(q w) = fma(q + 128, w, -128 w)
    // exactly (the fma forms (q + 128) w - 128 w = q w before its one rounding).
    float2 u[kQ];        // a_CB dt_i exp(r_I - cs_i)
    float2 dtcb[kQ];     // a_CB dt_i
    float csr[kQ];       // cs_i - r_{I-1} (r_{-1} = 0), fp32
    float eoff[kQ];      // a_C(j) exp(cs_j)
    float R[8][8];       // exp(r_a - r_b), b <= a
    float aS[kP];
    float cr[kP];
    double cs[kQ];
    double scan[4];
    // x^T [p][i] fp16 (the ChunkScan2 MFMA operand) and, for fp16 x, x in row order [j][p] (the
    // D skip operand), which the epilogue overwrites in place with y as the output stage.
    uint8_t xT[kP * kXTS];
    uint8_t xr[kHalfX ? kQ * kYS : 16];
  };
  __shared__ Smem sm;
  float2* s_u = sm.u;
  float2* s_dtcb = sm.dtcb;
  float* s_csr = sm.csr;
  float* s_eoff = sm.eoff;
  float (*s_R)[8] = sm.R;
  float* s_aS = sm.aS;
  float* s_cr = sm.cr;
  double* s_cs = sm.cs;
  double* s_scan = sm.scan;
  uint8_t* s_xT = sm.xT;
  uint8_t* s_xr = sm.xr;

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
  if (t < kP) {
    s_aS[t] = state_scale[h * kP + t];
    s_cr[t] = corr ? corr[h * kP + t] : 0.0f;
  }
  __syncthreads();
  {
    const int blk = t >> 5;
    const float dtcb = aCB * dtv;
    const float u = dtcb * expf((float)(s_cs[blk * 32 + 31] - cs));
    s_dtcb[t] = make_float2(dtcb, -128.0f * dtcb);
    s_u[t] = make_float2(u, -128.0f * u);
    s_csr[t] = (float)(blk ? cs - s_cs[blk * 32 - 1] : cs);
    const float ac = c_per_token ? C_scale[(tok0 + t) * G + g] : C_scale[g];
    s_eoff[t] = ac * expf((float)cs);
    if (t < 64) {
      const int ra = t >> 3, rb = t & 7;
      s_R[ra][rb] = (rb <= ra) ? expf((float)(s_cs[ra * 32 + 31] - s_cs[rb * 32 + 31])) : 0.0f;
    }
  }
  // ---- x^T [p][i] (fp16) and x rows [j][p] (fp16 input) in LDS
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
    if constexpr (kHalfX) {
#pragma unroll
      for (int r = 0; r < 32; ++r)
        *reinterpret_cast<uint32_t*>(s_xr + (jb * 32 + r) * kYS + p0 * 2) = (uint32_t)xr[r];
    }
  }
  __syncthreads();

  // Both products are formed transposed (MFMA rows = channels p, columns = tokens j), so each
  // lane owns one token row j and runs of 4 consecutive channels: the epilogue needs one row
  // factor per lane and moves 8-byte vectors.  Lane l: j = 32 jt + (l % 32); accumulator
  // register r holds channel p = 32 pt + 8 (r / 4) + 4 (l / 32) + r % 4.
  const int8_t* pbase = pin + (((size_t)b * nc + c) * H + h) * (size_t)kP * kN;
  const int8_t* cbbase = cbq + (((size_t)b * nc + c) * G + g) * (size_t)kQ * kQ;
  const int pc = lane & 31, half = lane >> 5;
  const float Dh = Dv ? Dv[h] : 0.0f;

  for (int q2 = 0; q2 < 2; ++q2) {
    const int jt = q2 ? 7 - wv : wv;
    const int jrow = jt * 32 + pc;
    // -- Scan1: Y1^T = P_in . C_q^T, int8 MFMA over n
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
        yi0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0[ks], a[ks], yi0, 0, 0, 0);
        yi1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1[ks], a[ks], yi1, 0, 0, 0);
      }
    }
    // -- Scan2: y_diag^T = x^T . W^T, fp16 MFMA over the causal source tokens i; CB_q of
    //    block it+1 is prefetched while block it is built
    v16f yd0 = {}, yd1 = {};
    {
      const int8_t* cbrow = cbbase + (size_t)jrow * kQ + 8 * half;
      const float csrj = s_csr[jrow];
      uint2 cur0 = *reinterpret_cast<const uint2*>(cbrow);
      uint2 cur1 = *reinterpret_cast<const uint2*>(cbrow + 16);
      for (int it = 0; it <= jt; ++it) {
        uint2 nx0 = cur0, nx1 = cur1;
        if (it < jt) {
          nx0 = *reinterpret_cast<const uint2*>(cbrow + (it + 1) * 32);
          nx1 = *reinterpret_cast<const uint2*>(cbrow + (it + 1) * 32 + 16);
        }
        // row factor of an off-diagonal block: exp(cs_j - r_{J-1}) exp(r_{J-1} - r_I)
        const float vj = (it < jt) ? __expf(csrj) * s_R[jt - 1][it] : 0.0f;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const uint2 cb8 = ks ? cur1 : cur0;
          const int i0 = it * 32 + ks * 16 + 8 * half;
          // int8 weights as unsigned bytes (q + 128), 4 per dword
          const uint32_t ub0 = cb8.x ^ 0x80808080u, ub1 = cb8.y ^ 0x80808080u;
          float wv[8];
          if (it < jt) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float2 uu = s_u[i0 + e];
              const float qb = (float)(((e < 4 ? ub0 : ub1) >> (8 * (e & 3))) & 0xffu);
              wv[e] = __builtin_fmaf(qb, uu.x, uu.y) * vj;
            }
          } else {
            // diagonal block: exp per element; the clamp keeps the masked (i > j) entries finite
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int i = i0 + e;
              const float2 dd = s_dtcb[i];
              const float qb = (float)(((e < 4 ? ub0 : ub1) >> (8 * (e & 3))) & 0xffu);
              const float ex = __expf(__builtin_fminf(csrj - s_csr[i], 0.0f));
              const float v = __builtin_fmaf(qb, dd.x, dd.y) * ex;
              wv[e] = (i <= jrow) ? v : 0.0f;
            }
          }
          v8h wf;
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            typedef float f2_t __attribute__((ext_vector_type(2)));
            typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
            const f2_t pr = {wv[e], wv[e + 1]};
            const h2_t hh = __builtin_convertvector(pr, h2_t);
            wf[e] = hh.x;
            wf[e + 1] = hh.y;
          }
          const v8h xa0 = *reinterpret_cast<const v8h*>(s_xT + pc * kXTS + i0 * 2);
          const v8h xa1 = *reinterpret_cast<const v8h*>(s_xT + (32 + pc) * kXTS + i0 * 2);
          yd0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(xa0, wf, yd0, 0, 0, 0);
          yd1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(xa1, wf, yd1, 0, 0, 0);
        }
        cur0 = nx0;
        cur1 = nx1;
      }
    }
    // -- epilogue of token row jrow: y = Y1 a_C exp(cs_j) a_S[p] + y_diag + D x + corr[p]
    const float eo = s_eoff[jrow];
    const size_t orow = (tok0 + jrow) * HP + (size_t)h * kP;
#pragma unroll
    for (int pt = 0; pt < 2; ++pt) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int pb = pt * 32 + 8 * g4 + 4 * half;
        const float4 as4 = *reinterpret_cast<const float4*>(s_aS + pb);
        const float4 cr4 = *reinterpret_cast<const float4*>(s_cr + pb);
        float xv[4];
        if constexpr (kHalfX) {
          const uint2 xw = *reinterpret_cast<const uint2*>(s_xr + jrow * kYS + pb * 2);
          xv[0] = (float)__builtin_bit_cast(_Float16, (uint16_t)(xw.x & 0xffffu));
          xv[1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(xw.x >> 16));
          xv[2] = (float)__builtin_bit_cast(_Float16, (uint16_t)(xw.y & 0xffffu));
          xv[3] = (float)__builtin_bit_cast(_Float16, (uint16_t)(xw.y >> 16));
        } else {
          const float4 xf = *reinterpret_cast<const float4*>(x + orow + pb);
          xv[0] = xf.x; xv[1] = xf.y; xv[2] = xf.z; xv[3] = xf.w;
        }
        const float asv[4] = {as4.x, as4.y, as4.z, as4.w};
        const float crv[4] = {cr4.x, cr4.y, cr4.z, cr4.w};
        float v[4];
        int yi[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r = 4 * g4 + q;
          yi[q] = pt ? yi1[r] : yi0[r];
          const float yd = pt ? yd1[r] : yd0[r];
          v[q] = (((float)yi[q] * eo) * asv[q] + yd) + Dh * xv[q] + crv[q];
        }
        if (y1_tap)
          *reinterpret_cast<int4*>(y1_tap + orow + pb) = make_int4(yi[0], yi[1], yi[2], yi[3]);
        if constexpr (sizeof(YT) == 4) {
          *reinterpret_cast<float4*>(y + orow + pb) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          uint2 o;
          o.x = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v[0]) |
                ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v[1]) << 16);
          o.y = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v[2]) |
                ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v[3]) << 16);
          if constexpr (kHalfX)
            *reinterpret_cast<uint2*>(s_xr + jrow * kYS + pb * 2) = o;   // in place over x
          else
            *reinterpret_cast<uint2*>(y + orow + pb) = o;
        }
      }
    }
  }

  if constexpr (sizeof(YT) == 2 && kHalfX) {
    __syncthreads();
#pragma unroll
    for (int k = 0; k < (kQ * kP * 2) / (16 * 256); ++k) {
      const int idx = k * 256 + t;
      const int j = idx >> 3, col = idx & 7;
      *reinterpret_cast<uint4*>(reinterpret_cast<uint8_t*>(y) +
                                ((tok0 + j) * HP + (size_t)h * kP) * 2 + col * 16) =
          *reinterpret_cast<const uint4*>(s_xr + j * kYS + col * 16);
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
