// ChunkBMM with INT8 operands (Sec. 4.2 "Quantization of ChunkBMM and ChunkScan2"):
//   CB32[j, i] = sum_n C_q[j, n] B_q[i, n]   for i <= j   (int8 MFMA, int32 accumulation)
//   CB_q[j, i] = clamp(rne(fl32(CB32) * m_CB[j]), -127, 127),  m_CB = fl32(a_C a_B / a_CB)
// Both operands are stored token-major with the contraction axis n contiguous, which is exactly
// the per-lane K-slice layout of v_mfma_i32_32x32x32_i8, so they feed the MFMA without a
// transpose.  B and C stay on the group axis (no broadcast to heads).
//
// The same workgroup also writes B_q^T of its chunk ([n][j], j contiguous): ChunkState contracts
// over tokens and needs B with the token axis contiguous, and every head of the group reuses it.
#include "common.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kBS = kN + 16;  // LDS row stride (bytes) of the staged B_q chunk

__global__ __launch_bounds__(256) void chunk_bmm_kernel(
    const int8_t* __restrict__ Cq, const int8_t* __restrict__ Bq,
    const float* __restrict__ C_scale, int c_per_token, const float* __restrict__ B_scale,
    const float* __restrict__ cb_scale, int8_t* __restrict__ cbq, int32_t* __restrict__ cb32_tap,
    int8_t* __restrict__ bqT, int L, int G, int nc) {
  __shared__ __attribute__((aligned(16))) int8_t s_b[kQ * kBS];
  __shared__ float s_m[kQ];

  const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int g = w % G;
  const int bc = w / G;
  const int c = bc % nc;
  const int b = bc / nc;
  const size_t tok0 = (size_t)b * L + (size_t)c * kQ;
  const size_t rs = (size_t)G * kN;  // token stride of B_q / C_q rows
  const int8_t* cbase = Cq + tok0 * rs + (size_t)g * kN;
  const int8_t* bbase = Bq + tok0 * rs + (size_t)g * kN;

  {  // requant multiplier per output row j (per-group, or per-token C step)
    const float ac = c_per_token ? C_scale[(tok0 + t) * G + g] : C_scale[g];
    s_m[t] = (float)(((double)ac * (double)B_scale[g]) / (double)cb_scale[g]);
  }
  // stage the B_q chunk (256 x 128 bytes), 16 bytes per thread per pass
#pragma unroll
  for (int it = 0; it < (kQ * kN) / (16 * 256); ++it) {
    const int idx = it * 256 + t;
    const int j = idx >> 3, col = (idx & 7) * 16;
    *reinterpret_cast<uint4*>(s_b + j * kBS + col) =
        *reinterpret_cast<const uint4*>(bbase + (size_t)j * rs + col);
  }
  __syncthreads();

  // B_q^T of this chunk: thread -> state index n (0..127), half of the tokens
  {
    const int n = t & 127, jh = t >> 7;
    int8_t* dstrow = bqT + ((((size_t)b * nc + c) * G + g) * kN + n) * kQ;
#pragma unroll
    for (int blk = 0; blk < kQ / 32; ++blk) {
      const int j0 = jh * (kQ / 2) + blk * 16;
      uint32_t wd[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        wd[u] = pack4_i8(s_b[(j0 + 4 * u) * kBS + n], s_b[(j0 + 4 * u + 1) * kBS + n],
                         s_b[(j0 + 4 * u + 2) * kBS + n], s_b[(j0 + 4 * u + 3) * kBS + n]);
      }
      *reinterpret_cast<uint4*>(dstrow + j0) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
    }
  }

  // causal 32x32 tiles (jt >= it): 36 tiles, round-robin over the 4 waves
  const size_t obase = (((size_t)b * nc + c) * G + g) * (size_t)kQ * kQ;
  for (int tile = wv; tile < 36; tile += 4) {
    int jt = 0, acc_t = tile;
    while (acc_t > jt) { acc_t -= jt + 1; ++jt; }
    const int it = acc_t;
    v16i acc = {};
    const int8_t* arow = cbase + (size_t)(jt * 32 + (lane & 31)) * rs;
    const int8_t* brow = s_b + (it * 32 + (lane & 31)) * kBS;
#pragma unroll
    for (int ks = 0; ks < kN / 32; ++ks) {
      const int kof = ks * 32 + 16 * (lane >> 5);
      const v4i a = *reinterpret_cast<const v4i*>(arow + kof);
      const v4i bb = *reinterpret_cast<const v4i*>(brow + kof);
      acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, bb, acc, 0, 0, 0);
    }
    const int i = it * 32 + (lane & 31);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int j = jt * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      const bool keep = i <= j;
      const int v = keep ? acc[r] : 0;
      cbq[obase + (size_t)j * kQ + i] = (int8_t)(keep ? requant_i8(v, s_m[j]) : 0);
      if (cb32_tap) cb32_tap[obase + (size_t)j * kQ + i] = v;
    }
  }
}

}  // namespace

hipError_t launch_chunk_bmm(const LayerDims& d, const int8_t* Cq, const int8_t* Bq,
                            const float* C_scale, int c_per_token, const float* B_scale,
                            const float* cb_scale, int8_t* cbq, int32_t* cb32_tap, int8_t* bqT,
                            hipStream_t st) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.ngroups;
  if (nwork == 0) return hipSuccess;
  hipLaunchKernelGGL(chunk_bmm_kernel, dim3((unsigned)nwork), dim3(256), 0, st, Cq, Bq, C_scale,
                     c_per_token, B_scale, cb_scale, cbq, cb32_tap, bqT, d.seqlen, d.ngroups,
                     d.nchunks);
  return hipGetLastError();
}

}  // namespace ssdi8
