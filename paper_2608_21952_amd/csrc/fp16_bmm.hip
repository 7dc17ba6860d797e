// FP16 baseline, ChunkBMM (Alg. 2 module 4 without quantization):
//   CB[j, i] = sum_n C[j, n] B[i, n]   for i <= j   (fp16 MFMA 32x32x16, fp32 accumulation)
// stored in fp32, as the 36 causal 32x32 blocks of each (b, c, g) in the fragment order in which
// ChunkScan2 builds its weights (frag::cb_inblock, in fp32 elements).  Like the INT8 ChunkBMM it
// also leaves the operands of the later kernels in fragment order (frag::k16_offset): C rows of
// the chunk (ChunkScan1, K = n) and B^T of the chunk (ChunkState, rows n, K = tokens).
// Work item = (b, c, g, role): roles 0..8 compute 4 causal tiles each (one per wave), role 9
// transposes B.
#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kTileWGs = 9;
constexpr int kRoles = kTileWGs + 1;
constexpr int kHalfTok = kQ / 2;       // tokens per transposer pass
constexpr int kBRow = kN * 2 + 16;     // LDS bytes per staged B row (fp16)
constexpr int kStS = 36;               // floats per row of a wave's 32x32 fp32 stage

typedef _Float16 h8 __attribute__((ext_vector_type(8)));

// 8 consecutive fp16 operand values from a fp16 or fp32 row.
template <typename T> __device__ __forceinline__ h8 load8(const T* p);
template <> __device__ __forceinline__ h8 load8<_Float16>(const _Float16* p) {
  return *reinterpret_cast<const h8*>(p);
}
template <> __device__ __forceinline__ h8 load8<float>(const float* p) {
  const float4 a = reinterpret_cast<const float4*>(p)[0];
  const float4 b = reinterpret_cast<const float4*>(p)[1];
  h8 r;
  r[0] = (_Float16)a.x; r[1] = (_Float16)a.y; r[2] = (_Float16)a.z; r[3] = (_Float16)a.w;
  r[4] = (_Float16)b.x; r[5] = (_Float16)b.y; r[6] = (_Float16)b.z; r[7] = (_Float16)b.w;
  return r;
}

template <typename T>
__global__ __launch_bounds__(256) void fp16_bmm_kernel(const T* __restrict__ C,
                                                       const T* __restrict__ B,
                                                       float* __restrict__ cb_frag,
                                                       _Float16* __restrict__ bT_frag,
                                                       _Float16* __restrict__ c_frag,
                                                       uint32_t* __restrict__ cb_amax, int L,
                                                       int G, int nc) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kHalfTok * kBRow];

  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int role = w % kRoles;
  const int bcg = w / kRoles;
  const int g = bcg % G;
  const int bc = bcg / G;
  const int c = bc % nc;
  const int b = bc / nc;
  const size_t tok0 = (size_t)b * L + (size_t)c * kQ;
  const size_t rs = (size_t)G * kN;
  const T* cbase = C + tok0 * rs + (size_t)g * kN;
  const T* bbase = B + tok0 * rs + (size_t)g * kN;
  const size_t cg = ((size_t)b * nc + c) * G + g;

  if (role == kTileWGs) {
    // ---- B^T of the chunk in two passes of 128 tokens: stage the rows as fp16, then each
    //      thread assembles 16-byte runs of 8 tokens of one channel n
    _Float16* dst = bT_frag + cg * (size_t)kN * kQ;
    for (int pass = 0; pass < 2; ++pass) {
      const int j0p = pass * kHalfTok;
#pragma unroll
      for (int k = 0; k < (kHalfTok * kN) / (8 * 256); ++k) {
        const int idx = k * 256 + t;
        const int j = idx >> 4, col = (idx & 15) * 8;
        *reinterpret_cast<h8*>(smem + j * kBRow + col * 2) =
            load8<T>(bbase + (size_t)(j0p + j) * rs + col);
      }
      __syncthreads();
#pragma unroll
      for (int k = 0; k < (kHalfTok / 8) * kN / 256; ++k) {
        const int unit = k * 256 + t;
        const int n = unit & (kN - 1), jg = unit >> 7;   // channel, group of 8 tokens
        h8 v;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          v[e] = *reinterpret_cast<const _Float16*>(smem + (jg * 8 + e) * kBRow + n * 2);
        *reinterpret_cast<h8*>(dst + frag::k16_offset(n, j0p + jg * 8, kQ)) = v;
      }
      __syncthreads();
    }
    return;
  }

  // ---- one causal 32x32 tile per wave: CB^T tile = B_tile . C_tile^T (rows i, columns j)
  int jt = 0, it = role * 4 + wv;
  while (it > jt) { it -= jt + 1; ++jt; }
  const int half = lane >> 5;
  const T* crow = cbase + (size_t)(jt * 32 + (lane & 31)) * rs + 8 * half;
  const T* brow = bbase + (size_t)(it * 32 + (lane & 31)) * rs + 8 * half;
  h8 cf[kN / 16], bf[kN / 16];
#pragma unroll
  for (int ks = 0; ks < kN / 16; ++ks) {
    cf[ks] = load8<T>(crow + 16 * ks);
    bf[ks] = load8<T>(brow + 16 * ks);
  }
  if (it == 0) {
    // the C rows of block jt in ChunkScan1 fragment order (before the MFMA chain, so that no
    // branch separates the last MFMA from the reads of its result)
    _Float16* cdst = c_frag + cg * (size_t)kQ * kN;
#pragma unroll
    for (int ks = 0; ks < kN / 16; ++ks)
      *reinterpret_cast<h8*>(cdst + frag::k16_offset(jt * 32 + (lane & 31), 16 * ks + 8 * half,
                                                     kN)) = cf[ks];
  }
  v16f acc = {};
#pragma unroll
  for (int ks = 0; ks < kN / 16; ++ks)
    acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(bf[ks], cf[ks], acc, 0, 0, 0);
  // acc[r]: column j = lane % 32, row i = 8 (r / 4) + 4 half + r % 4; stage [j][i], then each
  // lane reads its ChunkScan2 K-slices i = 16 ks + 8 half + e of row j
  float* st = reinterpret_cast<float*>(smem) + wv * 32 * kStS;
  const int jj = lane & 31;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int ii = 8 * (r >> 2) + 4 * half + (r & 3);
    const bool keep = it < jt || ii <= jj;
    st[jj * kStS + ii] = keep ? acc[r] : 0.0f;
  }
  __syncthreads();
  float4 o[4];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    o[2 * ks] = *reinterpret_cast<const float4*>(st + jj * kStS + 16 * ks + 8 * half);
    o[2 * ks + 1] = *reinterpret_cast<const float4*>(st + jj * kStS + 16 * ks + 8 * half + 4);
  }
  float4* out = reinterpret_cast<float4*>(cb_frag + (cg * frag::kCbBlocks + frag::cb_block(jt, it)) *
                                          1024 + lane * 16);
#pragma unroll
  for (int u = 0; u < 4; ++u) out[u] = o[u];
  if (cb_amax) {
    // calibration: absolute maximum of the causal entries of this group's C.B^T (the masked
    // entries were staged as 0); bit patterns of non-negative floats order like the floats
    float m = 0.0f;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      m = __builtin_fmaxf(m, __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(o[u].x),
                                                             __builtin_fabsf(o[u].y)),
                                             __builtin_fmaxf(__builtin_fabsf(o[u].z),
                                                             __builtin_fabsf(o[u].w))));
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = __builtin_fmaxf(m, __shfl_xor(m, off, 64));
    if (lane == 0) atomicMax(cb_amax + g, __float_as_uint(m));
  }
}

}  // namespace

hipError_t launch_fp16_bmm(const LayerDims& d, const void* C, const void* B, int dtype,
                           float* cb_frag, _Float16* bT_frag, _Float16* c_frag,
                           uint32_t* cb_amax, hipStream_t st) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.ngroups * kRoles;
  if (nwork == 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(fp16_bmm_kernel<_Float16>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const _Float16*>(C), static_cast<const _Float16*>(B),
                       cb_frag, bT_frag, c_frag, cb_amax, d.seqlen, d.ngroups, d.nchunks);
  else
    hipLaunchKernelGGL(fp16_bmm_kernel<float>, dim3((unsigned)nwork), dim3(256), 0, st,
                       static_cast<const float*>(C), static_cast<const float*>(B), cb_frag,
                       bT_frag, c_frag, cb_amax, d.seqlen, d.ngroups, d.nchunks);
  return hipGetLastError();
}

}  // namespace ssdi8
