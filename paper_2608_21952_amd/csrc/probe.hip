// On-box peak of the matrix cores: every wave runs four independent MFMA accumulation chains
// (enough to cover the instruction latency) on register operands, so the loop is bound by the
// MFMA issue rate alone.  The measured rate is the denominator a "fraction of measured peak"
// uses next to the datasheet figure.
#include "common.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kChains = 4;

__global__ __launch_bounds__(256) void mfma_i8_loop(int64_t iters, int32_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const v4i a = {lane, lane + 1, lane + 2, lane + 3};
  const v4i b = {3 - lane, 2 - lane, 1 - lane, -lane};
  v16i c[kChains] = {};
  for (int64_t i = 0; i < iters; ++i) {
#pragma unroll
    for (int k = 0; k < kChains; ++k) c[k] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c[k], 0, 0, 0);
  }
  int32_t s = 0;
#pragma unroll
  for (int k = 0; k < kChains; ++k) s += c[k][0] + c[k][15];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void mfma_f16_loop(int64_t iters, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  v8h a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (_Float16)(0.001f * (float)(lane + e));
    b[e] = (_Float16)(0.001f * (float)(e - lane));
  }
  v16f c[kChains] = {};
  for (int64_t i = 0; i < iters; ++i) {
#pragma unroll
    for (int k = 0; k < kChains; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c[k], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < kChains; ++k) s += c[k][0] + c[k][15];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

}  // namespace

int64_t mfma_probe_ops(int dtype, int64_t iters, int64_t blocks) {
  const int64_t per = dtype == 0 ? 32 * 32 * 32 * 2 : 32 * 32 * 16 * 2;
  return blocks * 4 /* waves */ * iters * kChains * per;
}

hipError_t launch_mfma_probe(int dtype, int64_t iters, int64_t blocks, void* out, hipStream_t st) {
  if (dtype == 0)
    hipLaunchKernelGGL(mfma_i8_loop, dim3((unsigned)blocks), dim3(256), 0, st, iters,
                       static_cast<int32_t*>(out));
  else
    hipLaunchKernelGGL(mfma_f16_loop, dim3((unsigned)blocks), dim3(256), 0, st, iters,
                       static_cast<float*>(out));
  return hipGetLastError();
}

}  // namespace ssdi8
