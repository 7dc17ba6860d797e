// Activation quantization (Eq. 1): static steps, or dynamic absmax/127 steps per granule.
// Used for B and C once per layer along the group axis (Sec. 4.2) and, in TOKEN mode, for
// per-token C steps (one wavefront reduction per token row).
#include "common.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

template <typename T>
__device__ __forceinline__ float ld_f32(const T* p, int64_t i) {
  return (float)p[i];
}

__device__ __forceinline__ int64_t granule_of(int64_t e, int gran, int64_t k, int64_t m) {
  int64_t row = e / m;
  switch (gran) {
    case 0: return 0;                // tensor
    case 1: return row % k;          // group
    case 2: return e % (k * m);      // channel
    default: return row;             // token
  }
}

// 16 consecutive elements per thread; requires m % 16 == 0 (all 16 share one (b,l,k) row).
// I is the index type: 32-bit whenever the element count allows (no 64-bit divisions).
template <typename T, typename I>
__global__ __launch_bounds__(256) void quant_static_vec16(const T* __restrict__ src,
                                                          int8_t* __restrict__ dst,
                                                          const float* __restrict__ scale,
                                                          int gran, I nvec, I k, I m) {
  const I rowvecs = m / 16;
  for (I v = (I)blockIdx.x * blockDim.x + threadIdx.x; v < nvec; v += (I)gridDim.x * blockDim.x) {
    const I e0 = v * 16;
    float x[16];
    if constexpr (sizeof(T) == 2) {
      const uint4* s = reinterpret_cast<const uint4*>(src + e0);
      uint4 a = s[0], b = s[1];
      const _Float16* ha = reinterpret_cast<const _Float16*>(&a);
      const _Float16* hb = reinterpret_cast<const _Float16*>(&b);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        x[i] = (float)ha[i];
        x[8 + i] = (float)hb[i];
      }
    } else {
      const float4* s = reinterpret_cast<const float4*>(src + e0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float4 f = s[i];
        x[4 * i] = f.x; x[4 * i + 1] = f.y; x[4 * i + 2] = f.z; x[4 * i + 3] = f.w;
      }
    }
    const I row = v / rowvecs;
    uint32_t q[16];
    if (gran == 2) {
      const I c0 = (row % k) * m + (v - row * rowvecs) * 16;   // channel of element 0
#pragma unroll
      for (int i = 0; i < 16; ++i) q[i] = quant_bits(x[i], 1.0f / scale[c0 + i]);
    } else {
      const I gi = gran == 0 ? 0 : (gran == 1 ? row % k : row);
      const float inv = 1.0f / scale[gi];
#pragma unroll
      for (int i = 0; i < 16; ++i) q[i] = quant_bits(x[i], inv);
    }
    uint4 o;
    o.x = pack_lo4(q[0], q[1], q[2], q[3]);
    o.y = pack_lo4(q[4], q[5], q[6], q[7]);
    o.z = pack_lo4(q[8], q[9], q[10], q[11]);
    o.w = pack_lo4(q[12], q[13], q[14], q[15]);
    *reinterpret_cast<uint4*>(dst + e0) = o;
  }
}

// fp16 source, m % 8 == 0: units of 8 consecutive elements (one 16-byte load, one 8-byte
// store), lane-contiguous so that a wave's loads cover one contiguous 1 KB; kU units per thread
// in flight.  32-bit indices (n < 2^31).
template <int kU>
__global__ __launch_bounds__(256) void quant_static_h8(const _Float16* __restrict__ src,
                                                      int8_t* __restrict__ dst,
                                                      const float* __restrict__ scale, int gran,
                                                      uint32_t nunit, uint32_t k, uint32_t m) {
  const uint32_t rowunits = m / 8;
  const uint32_t u0 = blockIdx.x * (256u * kU) + threadIdx.x;
  uint4 raw[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const uint32_t unit = u0 + 256u * u;
    if (unit < nunit) raw[u] = reinterpret_cast<const uint4*>(src)[unit];
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const uint32_t unit = u0 + 256u * u;
    if (unit >= nunit) break;
    const uint32_t row = unit / rowunits;
    const uint32_t w[4] = {raw[u].x, raw[u].y, raw[u].z, raw[u].w};
    uint32_t q[8];
    if (gran == 2) {
      const uint32_t c0 = (row % k) * m + (unit - row * rowunits) * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float x = (float)__builtin_bit_cast(
            _Float16, (uint16_t)((i & 1) ? (w[i >> 1] >> 16) : (w[i >> 1] & 0xffffu)));
        q[i] = quant_bits(x, 1.0f / scale[c0 + i]);
      }
    } else {
      const uint32_t gi = gran == 0 ? 0u : (gran == 1 ? row % k : row);
      const float inv = 1.0f / scale[gi];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float x = (float)__builtin_bit_cast(
            _Float16, (uint16_t)((i & 1) ? (w[i >> 1] >> 16) : (w[i >> 1] & 0xffffu)));
        q[i] = quant_bits(x, inv);
      }
    }
    reinterpret_cast<uint2*>(dst)[unit] =
        make_uint2(pack_lo4(q[0], q[1], q[2], q[3]), pack_lo4(q[4], q[5], q[6], q[7]));
  }
}

template <typename T>
__global__ __launch_bounds__(256) void quant_static_scalar(const T* __restrict__ src,
                                                           int8_t* __restrict__ dst,
                                                           const float* __restrict__ scale,
                                                           int gran, int64_t n, int64_t k,
                                                           int64_t m) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    dst[e] = (int8_t)quant_i8(ld_f32(src, e), 1.0f / scale[granule_of(e, gran, k, m)]);
  }
}

__global__ void fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// Absolute maximum per granule (tensor / group / channel, at most kMaxGranules granules),
// accumulated as the bit patterns of non-negative floats (their integer order is the float
// order) with LDS and then global atomic max into `acc` (pre-zeroed).
constexpr int kMaxGranules = 8192;

template <typename T>
__global__ __launch_bounds__(256) void absmax_granules(const T* __restrict__ src,
                                                       uint32_t* __restrict__ acc, int gran,
                                                       int64_t n, int64_t k, int64_t m,
                                                       int ngran) {
  __shared__ uint32_t smax[kMaxGranules];
  for (int i = threadIdx.x; i < ngran; i += blockDim.x) smax[i] = 0u;
  __syncthreads();
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    float a = __builtin_fabsf(ld_f32(src, e));
    atomicMax(&smax[granule_of(e, gran, k, m)], __float_as_uint(a));
  }
  __syncthreads();
  for (int i = threadIdx.x; i < ngran; i += blockDim.x)
    if (smax[i]) atomicMax(&acc[i], smax[i]);
}

// The same absmax when the k m values of a (b, l) row split into 16-byte units of kE elements
// that never straddle two granules (m % kE == 0): the rows are the outer loop and each thread
// owns fixed units (columns) of them, so the granule of each of its values never changes and
// its running maxima stay in registers (kE of them per column for CHANNEL, one otherwise).
// A block is TR rows x TC columns of threads.  When a thread leaves a column, the lanes of one
// granule first combine their maxima by shuffles (gsz consecutive lanes: m / kE for GROUP, the
// whole wave for TENSOR, one lane for CHANNEL), so that one lane per granule and wave updates
// LDS.  Each block then writes its ngran maxima to part[block] (all of them, zeros included),
// which absmax_partials_to_step reduces; or, with part NULL, updates each global word of `acc`
// once by atomic max.
template <typename T>
__global__ __launch_bounds__(256) void absmax_cols(const T* __restrict__ src,
                                                   uint32_t* __restrict__ acc,
                                                   uint32_t* __restrict__ part, int gran,
                                                   int64_t rows, int cols, int tc, int m,
                                                   int ngran, int gsz) {
  constexpr int kE = 16 / sizeof(T);
  __shared__ uint32_t smax[kMaxGranules];
  for (int i = threadIdx.x; i < ngran; i += blockDim.x) smax[i] = 0u;
  __syncthreads();
  const int tx = threadIdx.x % tc, ty = threadIdx.x / tc, tr = blockDim.x / tc;
  const int lane = threadIdx.x & 63;
  for (int col0 = 0; col0 < cols; col0 += tc) {
    const int col = col0 + tx;
    const bool live = col < cols;
    float mx[kE];
#pragma unroll
    for (int e = 0; e < kE; ++e) mx[e] = 0.0f;
    if (live) {
#pragma unroll 4
      for (int64_t row = (int64_t)blockIdx.x * tr + ty; row < rows;
           row += (int64_t)gridDim.x * tr) {
        const uint4 u = reinterpret_cast<const uint4*>(src + (row * cols + col) * kE)[0];
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
        if constexpr (sizeof(T) == 2) {
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            const float v = (float)__builtin_bit_cast(
                _Float16, (uint16_t)((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu)));
            mx[e] = __builtin_fmaxf(mx[e], __builtin_fabsf(v));
          }
        } else {
#pragma unroll
          for (int e = 0; e < kE; ++e)
            mx[e] = __builtin_fmaxf(mx[e], __builtin_fabsf(__uint_as_float(w[e])));
        }
      }
    }
    if (gran == 2) {
      if (live) {
#pragma unroll
        for (int e = 0; e < kE; ++e)
          if (mx[e] > 0.0f) atomicMax(&smax[col * kE + e], __float_as_uint(mx[e]));
      }
    } else {
      float v = mx[0];
#pragma unroll
      for (int e = 1; e < kE; ++e) v = __builtin_fmaxf(v, mx[e]);
      // lanes of one granule are gsz consecutive lanes starting at a multiple of gsz
      for (int o = gsz >> 1; o > 0; o >>= 1) v = __builtin_fmaxf(v, __shfl_xor(v, o, 64));
      const int gi = gran == 0 ? 0 : (col * kE) / m;
      if (live && (lane & (gsz - 1)) == 0 && v > 0.0f) atomicMax(&smax[gi], __float_as_uint(v));
    }
  }
  __syncthreads();
  if (part) {
    for (int i = threadIdx.x; i < ngran; i += blockDim.x)
      part[(size_t)blockIdx.x * ngran + i] = smax[i];
  } else {
    for (int i = threadIdx.x; i < ngran; i += blockDim.x)
      if (smax[i]) atomicMax(&acc[i], smax[i]);
  }
}

// step[g] = max over blocks of part[block][g] (float bits) / 127, or 1 for an all-zero granule
// (as absmax_to_step): one block per granule.
__global__ __launch_bounds__(256) void absmax_partials_to_step(const uint32_t* __restrict__ part,
                                                               int nblocks, int ngran,
                                                               float* __restrict__ scale) {
  __shared__ uint32_t wmax[4];
  const int g = blockIdx.x;
  uint32_t v = 0u;
  for (int b = threadIdx.x; b < nblocks; b += blockDim.x) {
    const uint32_t x = part[(size_t)b * ngran + g];
    v = x > v ? x : v;
  }
  for (int o = 32; o > 0; o >>= 1) {
    const uint32_t x = (uint32_t)__shfl_xor((int)v, o, 64);
    v = x > v ? x : v;
  }
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) v = wmax[w] > v ? wmax[w] : v;
    v = wmax[0] > v ? wmax[0] : v;
    const float a = __uint_as_float(v) / 127.0f;
    scale[g] = (a == 0.0f) ? 1.0f : a;
  }
}

__global__ void absmax_to_step(float* scale, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    float a = __uint_as_float(__float_as_uint(scale[i])) / 127.0f;
    scale[i] = (a == 0.0f) ? 1.0f : a;
  }
}

// TOKEN granularity, dynamic: one wavefront per (b,l,k) row of m elements.
template <typename T>
__global__ __launch_bounds__(256) void quant_token_dynamic(const T* __restrict__ src,
                                                           int8_t* __restrict__ dst,
                                                           float* __restrict__ scale,
                                                           int64_t rows, int64_t m) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T* s = src + row * m;
  float mx = 0.0f;
  for (int64_t i = lane; i < m; i += 64) mx = __builtin_fmaxf(mx, __builtin_fabsf((float)s[i]));
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) mx = __builtin_fmaxf(mx, __shfl_xor(mx, off, 64));
  float a = mx / 127.0f;
  a = (a == 0.0f) ? 1.0f : a;
  if (lane == 0) scale[row] = a;
  const float inv = 1.0f / a;
  for (int64_t i = lane; i < m; i += 64) dst[row * m + i] = (int8_t)quant_i8((float)s[i], inv);
}

// blocks of the dynamic absmax (several per CU for loads in flight; their partial maxima are
// reduced by a second kernel, so more blocks cost no atomics)
constexpr int64_t kAbsmaxBlocks = 512;

inline int64_t grid_for(int64_t items, int per_block = 256, int64_t cap = 65536) {
  int64_t g = (items + per_block - 1) / per_block;
  return g < 1 ? 1 : (g > cap ? cap : g);
}

template <typename T>
hipError_t quantize_impl(const T* src, int64_t b, int64_t l, int64_t k, int64_t m, int gran,
                         float* scale, int compute_scale, int8_t* dst, hipStream_t st) {
  const int64_t n = b * l * k * m;
  if (compute_scale && gran == 3) {
    const int64_t rows = b * l * k;
    if (rows == 0) return hipSuccess;
    hipLaunchKernelGGL(quant_token_dynamic<T>, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0,
                       st, src, dst, scale, rows, m);
    return hipGetLastError();
  }
  if (compute_scale) {
    const int ngran = gran == 0 ? 1 : (gran == 1 ? (int)k : (int)(k * m));
    constexpr int kE = 16 / sizeof(T);
    const int64_t cols = k * m / kE;
    if (n > 0 && m % kE == 0 && cols <= ((int64_t)1 << 20)) {
      // columns of 16-byte units, rows of b l: a wave spans up to 64 consecutive units of a row
      const int tc = cols < 64 ? (int)cols : 64;
      const int tr = 256 / tc;
      const int64_t rows = b * l;
      // lanes sharing a granule: the wave (TENSOR, when a wave holds columns of one row only),
      // the m / kE lanes of one group (GROUP, when that is a power of two dividing tc), else one
      int gsz = 1;
      const int upr = (int)(m / kE);   // units per granule row for GROUP
      if (gran == 0 && tc == 64) gsz = 64;
      if (gran == 1 && upr > 0 && (upr & (upr - 1)) == 0 && tc % upr == 0) gsz = upr;
      // the blocks' partial maxima go to dst, which holds nothing yet (it is written by the
      // quantization that follows), when they fit there; else one atomic max per block
      int64_t nb = grid_for(rows, tr, kAbsmaxBlocks);
      const int64_t room = n / (4 * (int64_t)ngran);
      if (room >= 1) {
        if (nb > room) nb = room;
        uint32_t* part = reinterpret_cast<uint32_t*>(dst);
        hipLaunchKernelGGL(absmax_cols<T>, dim3((unsigned)nb), dim3(256), 0, st, src, nullptr,
                           part, gran, rows, (int)cols, tc, (int)m, ngran, gsz);
        hipLaunchKernelGGL(absmax_partials_to_step, dim3((unsigned)ngran), dim3(256), 0, st,
                           part, (int)nb, ngran, scale);
      } else {
        hipLaunchKernelGGL(fill_u32, dim3((unsigned)grid_for(ngran)), dim3(256), 0, st,
                           reinterpret_cast<uint32_t*>(scale), (int64_t)ngran, 0u);
        hipLaunchKernelGGL(absmax_cols<T>, dim3((unsigned)grid_for(rows, tr, 256)), dim3(256), 0,
                           st, src, reinterpret_cast<uint32_t*>(scale), nullptr, gran, rows,
                           (int)cols, tc, (int)m, ngran, gsz);
        hipLaunchKernelGGL(absmax_to_step, dim3((unsigned)((ngran + 255) / 256)), dim3(256), 0,
                           st, scale, ngran);
      }
    } else {
      hipLaunchKernelGGL(fill_u32, dim3((unsigned)grid_for(ngran)), dim3(256), 0, st,
                         reinterpret_cast<uint32_t*>(scale), (int64_t)ngran, 0u);
      if (n > 0)
        hipLaunchKernelGGL(absmax_granules<T>, dim3((unsigned)grid_for(n, 256, 2048)), dim3(256),
                           0, st, src, reinterpret_cast<uint32_t*>(scale), gran, n, k, m, ngran);
      hipLaunchKernelGGL(absmax_to_step, dim3((unsigned)((ngran + 255) / 256)), dim3(256), 0, st,
                         scale, ngran);
    }
  }
  if (n == 0) return hipGetLastError();
  if (sizeof(T) == 2 && m % 8 == 0 && n < ((int64_t)1 << 31)) {
    constexpr int kU = 4;
    const int64_t nunit = n / 8;
    hipLaunchKernelGGL(quant_static_h8<kU>, dim3((unsigned)((nunit + 256 * kU - 1) / (256 * kU))),
                       dim3(256), 0, st, reinterpret_cast<const _Float16*>(src), dst, scale, gran,
                       (uint32_t)nunit, (uint32_t)k, (uint32_t)m);
  } else if (m % 16 == 0) {
    const int64_t nvec = n / 16;
    if (n < ((int64_t)1 << 31)) {
      hipLaunchKernelGGL((quant_static_vec16<T, uint32_t>), dim3((unsigned)grid_for(nvec)),
                         dim3(256), 0, st, src, dst, scale, gran, (uint32_t)nvec, (uint32_t)k,
                         (uint32_t)m);
    } else {
      hipLaunchKernelGGL((quant_static_vec16<T, uint64_t>), dim3((unsigned)grid_for(nvec)),
                         dim3(256), 0, st, src, dst, scale, gran, (uint64_t)nvec, (uint64_t)k,
                         (uint64_t)m);
    }
  } else {
    hipLaunchKernelGGL(quant_static_scalar<T>, dim3((unsigned)grid_for(n)), dim3(256), 0, st,
                       src, dst, scale, gran, n, k, m);
  }
  return hipGetLastError();
}

}  // namespace

int quantize_max_granules() { return kMaxGranules; }

hipError_t launch_quantize(const void* src, int src_dtype, int64_t b, int64_t l, int64_t k,
                           int64_t m, int gran, float* scale, int compute_scale, int8_t* dst,
                           hipStream_t st) {
  if (src_dtype == 1)
    return quantize_impl(static_cast<const _Float16*>(src), b, l, k, m, gran, scale,
                         compute_scale, dst, st);
  return quantize_impl(static_cast<const float*>(src), b, l, k, m, gran, scale, compute_scale,
                       dst, st);
}

}  // namespace ssdi8
