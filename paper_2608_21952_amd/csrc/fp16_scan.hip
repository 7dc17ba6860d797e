// FP16 baseline, ChunkScan1 + ChunkScan2 + output (Alg. 2 modules 5-6 without quantization):
//   Scan1  Y1[j, p] = sum_n C[j, n] fp16(P_in[p, n])      fp16 MFMA, fp32 accumulation
//   Scan2  W[j, i]  = fp16(CB[j, i] dt_i exp(cs_j - cs_i)), i <= j;  y_diag = W . x
//   y = Y1 exp(cs_j) + y_diag + D x
// The structure is the INT8 ChunkScan's (one workgroup per (b, c, h), transposed products so a
// lane owns a token row, x^T staged once in LDS, block-factorised decay, fp16 output staged
// through LDS), with fp32 CB blocks and fp32 entering states in place of the int8 ones.
#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kXTS = kQ * 2 + 16;
constexpr float kDiagSpan = 64.0f;
static_assert(kP * kXTS >= kQ * kP * 2, "the fp16 output stage reuses the x^T bytes");

template <typename XT> struct Pair;
template <> struct Pair<_Float16> {
  typedef uint32_t raw;
  template <int kPol = 0>
  static __device__ __forceinline__ raw load(__amdgpu_buffer_rsrc_t r, uint32_t vo, uint32_t so) {
    return buf_load4<kPol>(r, vo, so);
  }
  static __device__ __forceinline__ uint16_t lo(raw v) { return (uint16_t)(v & 0xffffu); }
  static __device__ __forceinline__ uint16_t hi(raw v) { return (uint16_t)(v >> 16); }
};
template <> struct Pair<float> {
  typedef float2 raw;
  template <int kPol = 0>
  static __device__ __forceinline__ raw load(__amdgpu_buffer_rsrc_t r, uint32_t vo, uint32_t so) {
    const uint2 v = buf_load8<kPol>(r, vo, so);
    return make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
  }
  static __device__ __forceinline__ uint16_t lo(raw v) {
    return __builtin_bit_cast(uint16_t, (_Float16)v.x);
  }
  static __device__ __forceinline__ uint16_t hi(raw v) {
    return __builtin_bit_cast(uint16_t, (_Float16)v.y);
  }
};

// 8 fp32 -> 8 fp16
__device__ __forceinline__ v8h to_h8(uint4 a, uint4 b) {
  typedef float f2_t __attribute__((ext_vector_type(2)));
  typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
  const float f[8] = {__uint_as_float(a.x), __uint_as_float(a.y), __uint_as_float(a.z),
                      __uint_as_float(a.w), __uint_as_float(b.x), __uint_as_float(b.y),
                      __uint_as_float(b.z), __uint_as_float(b.w)};
  v8h r;
#pragma unroll
  for (int e = 0; e < 8; e += 2) {
    const h2_t hh = __builtin_convertvector((f2_t){f[e], f[e + 1]}, h2_t);
    r[e] = hh.x;
    r[e + 1] = hh.y;
  }
  return r;
}

template <typename XT, typename YT>
__global__ __launch_bounds__(256, 3) void fp16_scan_kernel(
    const XT* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const _Float16* __restrict__ c_frag, const float* __restrict__ pin,
    const float* __restrict__ cb, const float* __restrict__ Dv, int dt_softplus,
    YT* __restrict__ y, int L, int H, int G, int nc, int stream) {
  struct __attribute__((aligned(16))) Smem {
    float u[kQ];         // dt_i exp(r_I - cs_i)                          (off-diagonal blocks)
    float dg[kQ];        // dt_i exp(r_{I-1} - cs_i) if block I has a small span, else dt_i
    float csr[kQ];       // cs_i - r_{I-1}
    float R[8][8];       // exp(r_a - r_b), b <= a
    double r[8];
    double scan[kScanScratch];
    alignas(16) uint8_t xT[kP * kXTS];   // 128-bit accesses: 16-byte aligned explicitly
  };
  __shared__ Smem sm;
  float* s_u = sm.u;
  float* s_dg = sm.dg;
  float* s_csr = sm.csr;
  float (*s_R)[8] = sm.R;
  double* s_r = sm.r;
  uint8_t* s_xT = sm.xT;

  const int t = threadIdx.x, lane = t & 63;
  const int wv = __builtin_amdgcn_readfirstlane(t >> 6);
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
    const __amdgpu_buffer_rsrc_t xrs = buffer_rsrc(x + tok0 * HP + (size_t)h * kP);
    const uint32_t xo = (uint32_t)((jb * 32 * HP + p0) * sizeof(XT));
    // x and y streamed when they exceed the Infinity Cache, as in the INT8 layer's scan
    if (stream) {
#pragma unroll
      for (int r = 0; r < 32; ++r)
        xr[r] = Pair<XT>::template load<kPolicyNT>(xrs, xo, (uint32_t)(r * HP * sizeof(XT)));
    } else {
#pragma unroll
      for (int r = 0; r < 32; ++r) xr[r] = Pair<XT>::load(xrs, xo, (uint32_t)(r * HP * sizeof(XT)));
    }
  }

  float dtv = dt[(tok0 + t) * H + h];
  if (dt_softplus) dtv = softplus_f32(dtv);   // the dt of this layer's ChunkState
  const float dA = dtv * A[h];
  const double cs = block_scan_f64_256(dA, sm.scan, sm.u);
  if ((t & 31) == 31) s_r[t >> 5] = cs;
  __syncthreads();
  {
    const int blk = t >> 5;
    const double rprev = blk ? s_r[blk - 1] : 0.0;
    s_u[t] = dtv * expf((float)(s_r[blk] - cs));
    const float csr = (float)(cs - rprev);
    s_csr[t] = csr;
    const bool small_span = (float)(s_r[blk] - rprev) >= -kDiagSpan;
    s_dg[t] = small_span ? dtv * expf(__builtin_fminf(-csr, kDiagSpan)) : dtv;
    if (t < 64) {
      const int ra = t >> 3, rb = t & 7;
      s_R[ra][rb] = (rb <= ra) ? expf((float)(s_r[ra] - s_r[rb])) : 0.0f;
    }
  }
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

  // Lane l: token row j = 32 jt + l % 32; accumulator register r holds channel
  // p = 32 pt + 8 (r / 4) + 4 (l / 32) + r % 4 (as in the INT8 ChunkScan).
  const int pc = lane & 31, half = lane >> 5;
  const size_t cg = ((size_t)b * nc + c) * G + g;
  const __amdgpu_buffer_rsrc_t prs =
      buffer_rsrc(pin + (((size_t)b * nc + c) * H + h) * (size_t)kP * kN);
  const __amdgpu_buffer_rsrc_t cbrs = buffer_rsrc(cb + cg * (size_t)frag::kCbBlocks * 1024);
  const __amdgpu_buffer_rsrc_t cqrs = buffer_rsrc(c_frag + cg * (size_t)kQ * kN);
  const uint32_t lane16 = lane * 16, lane64 = lane * 64;
  const float Dh = Dv ? Dv[h] : 0.0f;
  uint2 y_first[8], y_second[8];

  auto jblock = [&](const int jt, uint2 (&yo)[8]) {
    asm volatile("" ::: "memory");
    const int jrow = jt * 32 + pc;
    const float csrj = s_csr[jrow];
    const float ej = __expf(csrj);
    const size_t orow = (tok0 + jrow) * HP + (size_t)h * kP;
    // -- the Scan2 accumulators start from D x
    v16f yd0, yd1;
#pragma unroll
    for (int pt = 0; pt < 2; ++pt) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int pb = pt * 32 + 8 * g4 + 4 * half;
        float xv[4];
        if constexpr (sizeof(XT) == 2) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            xv[q] = (float)*reinterpret_cast<const _Float16*>(s_xT + (pb + q) * kXTS + jrow * 2);
        } else {
          const float4 xf = *reinterpret_cast<const float4*>(x + orow + pb);
          xv[0] = xf.x; xv[1] = xf.y; xv[2] = xf.z; xv[3] = xf.w;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (pt) yd1[4 * g4 + q] = Dh * xv[q];
          else yd0[4 * g4 + q] = Dh * xv[q];
        }
      }
    }
    // -- Scan2 over the causal blocks (jt, it); fp32 CB block: 16 floats per lane
    {
      const uint32_t cbrow = frag::cb_block(jt, 0) * 4096;
      const bool diag_fast =
          __builtin_amdgcn_readfirstlane((int)(s_csr[jt * 32 + 31] >= -kDiagSpan)) != 0;
      auto mfma_block = [&](const float (&wv)[8], int i0) {
        v8h wf;
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          typedef float f2_t __attribute__((ext_vector_type(2)));
          typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
          const h2_t hh = __builtin_convertvector((f2_t){wv[e], wv[e + 1]}, h2_t);
          wf[e] = hh.x;
          wf[e + 1] = hh.y;
        }
        const v8h xa0 = *reinterpret_cast<const v8h*>(s_xT + pc * kXTS + i0 * 2);
        const v8h xa1 = *reinterpret_cast<const v8h*>(s_xT + (32 + pc) * kXTS + i0 * 2);
        yd0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(xa0, wf, yd0, 0, 0, 0);
        yd1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(xa1, wf, yd1, 0, 0, 0);
      };
      auto load_block = [&](uint32_t off, uint4 (&v)[4]) {
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = buf_load16(cbrs, lane64, off + 16 * u);
      };
      auto cbv = [](const uint4 (&v)[4], int k) {   // float k of this lane's 16
        const uint4 q = v[k >> 2];
        const uint32_t e = (k & 3) == 0 ? q.x : (k & 3) == 1 ? q.y : (k & 3) == 2 ? q.z : q.w;
        return __uint_as_float(e);
      };
      uint4 cur[4];
      load_block(cbrow, cur);
      for (int it = 0; it < jt; ++it) {
        uint4 nx[4];
        load_block(cbrow + (it + 1) * 4096, nx);
        __builtin_amdgcn_sched_barrier(0);
        const float vj = ej * s_R[jt - 1][it];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int i0 = it * 32 + ks * 16 + 8 * half;
          float wv[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) wv[e] = (cbv(cur, 8 * ks + e) * s_u[i0 + e]) * vj;
          mfma_block(wv, i0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) cur[u] = nx[u];
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int i0 = jt * 32 + ks * 16 + 8 * half;
        float wv[8];
        if (diag_fast) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float v = (cbv(cur, 8 * ks + e) * s_dg[i0 + e]) * ej;
            wv[e] = (i0 + e <= jrow) ? v : 0.0f;
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float ex = __expf(__builtin_fminf(csrj - s_csr[i0 + e], 0.0f));
            const float v = (cbv(cur, 8 * ks + e) * s_dg[i0 + e]) * ex;
            wv[e] = (i0 + e <= jrow) ? v : 0.0f;
          }
        }
        mfma_block(wv, i0);
      }
    }
    // -- Scan1: Y1^T = fp16(P_in) . C^T over n (8 K-steps of 16)
    v16f yi0 = {}, yi1 = {};
    {
      uint32_t lofs = lane * 32;
      asm volatile("" : "+v"(lofs));
      const uint32_t crow = jt * (kN / 16) * 1024;
#pragma unroll
      for (int ks = 0; ks < kN / 16; ++ks) {
        const v8h a = __builtin_bit_cast(v8h, buf_load16(cqrs, lane16, crow + 1024 * ks));
        const uint32_t o0 = ks * 2048, o1 = (kN / 16 + ks) * 2048;
        const v8h p0f = to_h8(buf_load16(prs, lofs, o0), buf_load16(prs, lofs, o0 + 16));
        const v8h p1f = to_h8(buf_load16(prs, lofs, o1), buf_load16(prs, lofs, o1 + 16));
        yi0 = __builtin_amdgcn_mfma_f32_32x32x16_f16(p0f, a, yi0, 0, 0, 0);
        yi1 = __builtin_amdgcn_mfma_f32_32x32x16_f16(p1f, a, yi1, 0, 0, 0);
      }
    }
    // -- epilogue: y = Y1 exp(cs_j) + (y_diag + D x),  exp(cs_j) = exp(cs_j - r_{J-1}) exp(r_{J-1})
    const float eo = ej * (jt ? __expf((float)s_r[jt - 1]) : 1.0f);
#pragma unroll
    for (int pt = 0; pt < 2; ++pt) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int pb = pt * 32 + 8 * g4 + 4 * half;
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r = 4 * g4 + q;
          v[q] = __builtin_fmaf(pt ? yi1[r] : yi0[r], eo, pt ? yd1[r] : yd0[r]);
        }
        if constexpr (sizeof(YT) == 4) {
          *reinterpret_cast<float4*>(y + orow + pb) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          typedef float f2_t __attribute__((ext_vector_type(2)));
          typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
          const h2_t h01 = __builtin_convertvector((f2_t){v[0], v[1]}, h2_t);
          const h2_t h23 = __builtin_convertvector((f2_t){v[2], v[3]}, h2_t);
          uint2 o = make_uint2(__builtin_bit_cast(uint32_t, h01), __builtin_bit_cast(uint32_t, h23));
          asm volatile("" : "+v"(o.x), "+v"(o.y));
          yo[4 * pt + g4] = o;
        }
      }
    }
  };
  jblock(wv, y_first);
  jblock(7 - wv, y_second);

  if constexpr (sizeof(YT) == 2) {
    __syncthreads();
    uint8_t* s_y = s_xT;
    {
      const uint32_t jx = pc & 7;
      uint8_t* r0 = s_y + (wv * 32 + pc) * 128 + 8 * half;
      uint8_t* r1 = s_y + ((7 - wv) * 32 + pc) * 128 + 8 * half;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint32_t so = (k ^ jx) * 16;
        *reinterpret_cast<uint2*>(r0 + so) = y_first[k];
        *reinterpret_cast<uint2*>(r1 + so) = y_second[k];
      }
    }
    __syncthreads();
    {
      const int jt8 = t >> 3, col = t & 7;
      const uint8_t* src = s_y + jt8 * 128 + ((col ^ (jt8 & 7)) * 16);
      const __amdgpu_buffer_rsrc_t yrs = buffer_rsrc(y + tok0 * HP + (size_t)h * kP);
      const uint32_t yo = (uint32_t)(jt8 * HP * 2 + col * 16);
      if (stream) {
#pragma unroll
        for (int k = 0; k < (kQ * kP * 2) / (16 * 256); ++k)
          buf_store16<kPolicyNT>(*reinterpret_cast<const uint4*>(src + k * 32 * 128), yrs, yo,
                                 (uint32_t)(k * 32 * HP * 2));
      } else {
#pragma unroll
        for (int k = 0; k < (kQ * kP * 2) / (16 * 256); ++k)
          buf_store16(*reinterpret_cast<const uint4*>(src + k * 32 * 128), yrs, yo,
                      (uint32_t)(k * 32 * HP * 2));
      }
    }
  }
}

}  // namespace

hipError_t launch_fp16_scan(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                            int dt_softplus, const float* A, const _Float16* c_frag,
                            const float* pin, const float* cb, const float* D, void* y,
                            int y_dtype, hipStream_t st) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.nheads;
  if (nwork == 0) return hipSuccess;
  const int stream = stream_xy(d, x_dtype == 1 ? 2 : 4, y_dtype == 1 ? 2 : 4);
#define SSDI8_F16SCAN_LAUNCH(XT, YT)                                                           \
  hipLaunchKernelGGL((fp16_scan_kernel<XT, YT>), dim3((unsigned)nwork), dim3(256), 0, st,       \
                     static_cast<const XT*>(x), dt, A, c_frag, pin, cb, D, dt_softplus,        \
                     static_cast<YT*>(y), d.seqlen, d.nheads, d.ngroups, d.nchunks, stream)
  if (x_dtype == 1 && y_dtype == 1) SSDI8_F16SCAN_LAUNCH(_Float16, _Float16);
  else if (x_dtype == 1) SSDI8_F16SCAN_LAUNCH(_Float16, float);
  else if (y_dtype == 1) SSDI8_F16SCAN_LAUNCH(float, _Float16);
  else SSDI8_F16SCAN_LAUNCH(float, float);
#undef SSDI8_F16SCAN_LAUNCH
  return hipGetLastError();
}

}  // namespace ssdi8
