// ChunkBMM with INT8 operands (Sec. 4.2 "Quantization of ChunkBMM and ChunkScan2"):
//   CB32[j, i] = sum_n C_q[j, n] B_q[i, n]   for i <= j   (int8 MFMA, int32 accumulation)
//   CB_q[j, i] = clamp(rne(fl32(CB32) * m_CB[j]), -127, 127),  m_CB = fl32(a_C a_B / a_CB)
// Workgroups of 8 waves; S of them per (batch, chunk, group) (S = 1, 2 or 4, more when the
// chunk-groups are too few to fill the GPU), each taking the causal 32x32 tiles of a range of
// row blocks jt.  A workgroup loads the rows its tiles need once (C rows of its blocks, B rows of
// blocks 0 .. its last), quantizes them once (when they arrive unquantized) and keeps them in
// LDS as int8 [256][128] tiles whose 16-byte chunks are XOR-swizzled by row, so that the MFMA
// operand reads (16 bytes per lane, 32 rows x 2 K-halves per wave) and the row writes are free
// of bank conflicts.  Its tiles are spread over the 8 waves; each is 4 MFMAs over n with the
// operands read straight from LDS in the per-lane K-slice layout of v_mfma_i32_32x32x32_i8,
// formed transposed (MFMA rows = source tokens i, columns = target tokens j) so that a lane holds
// one target row: one requant multiplier per lane, and its CB-order 16-byte slice is complete
// after one exchange of two dwords with the other half-wave.
//
// Outputs for the later kernels are written in MFMA fragment order (frag.hpp): a wave reads
// each operand fragment as one contiguous 1 KB run.
//   CB_q   the 36 causal 32x32 blocks of the chunk, as ChunkScan2 B-operand fragments
//   C_q    a fragment-order copy of the chunk's C_q rows (ChunkScan1 operand), written by the
//          waves of the i = 0 blocks, which hold exactly those fragments in registers
//   B_q^T  ChunkState contracts over tokens and needs B with the token axis as the K-slice
//          (every head of the group reuses it): read column-wise from the B_q tile in LDS, the
//          S workgroups of a chunk-group taking 8 / S token blocks each
// B and C may also arrive unquantized (fp16 / fp32) with static steps: each row is then quantized
// as it is loaded (the B/C quantization of Eq. 1 fused into this kernel, which is the only reader
// of the row-major B_q, C_q), with the arithmetic of ssdi8_quantize_act.
#include <hip/hip_ext.h>

#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;

// Byte offset of 16-byte chunk k (0..7) of row r in a [256][128] int8 LDS tile: the chunk index
// is XOR-ed with (r / 2) % 8, so that 16 consecutive rows read at one k hit 16 distinct groups of
// four banks.
__device__ __forceinline__ int swz(int r, int k) { return r * kN + ((k ^ ((r >> 1) & 7)) << 4); }

// 16 consecutive K values of a B or C row as int8: already quantized (int8_t), or quantized here
// from fp16 / fp32 with the static step exactly as ssdi8_quantize_act does (Eq. 1:
// clamp(rne(fl32(v * fl32(1 / step))))).
template <typename T> struct Row16;
template <> struct Row16<int8_t> {
  static __device__ __forceinline__ uint4 load(const int8_t* p, float) {
    return *reinterpret_cast<const uint4*>(p);
  }
};
template <> struct Row16<_Float16> {
  static __device__ __forceinline__ uint4 load(const _Float16* p, float inv) {
    const uint4 a = reinterpret_cast<const uint4*>(p)[0], b = reinterpret_cast<const uint4*>(p)[1];
    const uint32_t w[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t q[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t wd = w[2 * i + (e >> 1)];
        q[e] = quant_bits((float)__builtin_bit_cast(_Float16, (uint16_t)((e & 1) ? (wd >> 16)
                                                                                  : (wd & 0xffffu))),
                          inv);
      }
      o[i] = pack_lo4(q[0], q[1], q[2], q[3]);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
  }
};
template <> struct Row16<float> {
  static __device__ __forceinline__ uint4 load(const float* p, float inv) {
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float4 f = reinterpret_cast<const float4*>(p)[i];
      o[i] = pack_lo4(quant_bits(f.x, inv), quant_bits(f.y, inv), quant_bits(f.z, inv),
                      quant_bits(f.w, inv));
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
  }
};

// Row-block range [jlo, jhi) of part s of S (S = 1, 2, 4): 36 causal tiles split as 36 / 21 + 15 /
// 10 + 11 + 7 + 8, so that each part loads about half the rows or fewer.
__device__ __forceinline__ void part_range(int s, int S, int* jlo, int* jhi) {
  if (S == 1) { *jlo = 0; *jhi = 8; return; }
  if (S == 2) { *jlo = s ? 6 : 0; *jhi = s ? 8 : 6; return; }
  const int lo[4] = {0, 4, 6, 7}, hi[4] = {4, 6, 7, 8};
  *jlo = lo[s];
  *jhi = hi[s];
}

// Work item w -> (b, c, g, part); the S parts of a chunk-group are consecutive work items.
template <typename T>
__global__ __launch_bounds__(kThreads) void chunk_bmm_kernel(
    const T* __restrict__ Cq, const T* __restrict__ Bq,
    const float* __restrict__ C_scale, int c_per_token, const float* __restrict__ B_scale,
    const float* __restrict__ cb_scale, int8_t* __restrict__ cbq_frag,
    int8_t* __restrict__ cbq_tap, int32_t* __restrict__ cb32_tap, int8_t* __restrict__ bqT_frag,
    int8_t* __restrict__ cq_frag, int cq_perm, int* __restrict__ sync, int nsync,
    int* __restrict__ timeouts, int L, int G, int nc, int S) {
  __shared__ __attribute__((aligned(16))) int8_t s_c[kQ * kN];
  __shared__ __attribute__((aligned(16))) int8_t s_b[kQ * kN];
  __shared__ float s_m[kQ];

  const int t = threadIdx.x, lane = t & 63;
  const int wv = __builtin_amdgcn_readfirstlane(t >> 6);
  // clears the ticket and hand-off flags of the single-pass scan that follows in the stream
  for (int i = blockIdx.x * kThreads + t; i < nsync; i += gridDim.x * kThreads) sync[i] = 0;
  // and the caller's count of hand-off waits that ran out (0 after the separate kernels)
  if (timeouts && blockIdx.x == 0 && t == 0) *timeouts = 0;
  const int w = xcd_remap(blockIdx.x, gridDim.x);
  const int part = w % S;
  const int g = (w / S) % G;
  const int bc = w / S / G;
  const int c = bc % nc;
  const int b = bc / nc;
  const size_t tok0 = (size_t)b * L + (size_t)c * kQ;
  const size_t rs = (size_t)G * kN;  // token stride of B_q / C_q rows
  const T* cbase = Cq + tok0 * rs + (size_t)g * kN;
  const T* bbase = Bq + tok0 * rs + (size_t)g * kN;
  const size_t cg = ((size_t)b * nc + c) * G + g;   // chunk-group index

  int jlo, jhi;
  part_range(part, S, &jlo, &jhi);

  // ---- rows of C (blocks [jlo, jhi)) and B (blocks [0, jhi)) -> int8 LDS tiles: chunk item q =
  //      16 values (row q / 8, chunk q % 8)
  {
    // inverse steps for B, C given unquantized (per group; C per token with c_per_token)
    const float inv_b = sizeof(T) == 1 ? 1.0f : 1.0f / B_scale[g];
    const float inv_cg = (sizeof(T) == 1 || c_per_token) ? 1.0f : 1.0f / C_scale[g];
    const int c0 = jlo * 32 * 8, c1 = jhi * 32 * 8, b1 = jhi * 32 * 8;
    uint4 vc[4], vb[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int q = u * kThreads + t, j = q >> 3, k = q & 7;
      if (q >= c0 && q < c1) {
        float inv_c = inv_cg;
        if (sizeof(T) != 1 && c_per_token) inv_c = 1.0f / C_scale[(tok0 + j) * G + g];
        vc[u] = Row16<T>::load(cbase + (size_t)j * rs + 16 * k, inv_c);
      }
      if (q < b1) vb[u] = Row16<T>::load(bbase + (size_t)j * rs + 16 * k, inv_b);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int q = u * kThreads + t, j = q >> 3, k = q & 7;
      if (q >= c0 && q < c1) *reinterpret_cast<uint4*>(s_c + swz(j, k)) = vc[u];
      if (q < b1) *reinterpret_cast<uint4*>(s_b + swz(j, k)) = vb[u];
    }
  }
  // requant multiplier per output row (per group, or per token row of C)
  if (t < kQ) {
    const float ac = c_per_token ? C_scale[(tok0 + t) * G + g] : C_scale[g];
    s_m[t] = (float)(((double)ac * (double)B_scale[g]) / (double)cb_scale[g]);
  }
  __syncthreads();

  // ---- B_q^T of this part's token blocks [8 part / S, 8 (part + 1) / S) ([n][j]): units of
  //      4 channels n x 16 tokens j, one per thread: 16 dword reads (4 bytes of n per token row),
  //      four 4x4 byte transposes, then one 16-byte run of j per channel
  static_assert(kThreads * 64 == kQ * kN, "one 4 x 16 unit per thread for the whole chunk");
  if (t < kThreads / S) {
    int8_t* dst = bqT_frag + cg * (size_t)kN * kQ;
    const int n0 = 4 * (t & 31), j0 = 16 * (t >> 5) + (kQ / S) * part;
    const int nk = n0 >> 4, nb = n0 & 15;
    uint32_t col[4][4];   // [n - n0][4-token group]
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      uint32_t r[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = j0 + 4 * g4 + i;
        r[i] = *reinterpret_cast<const uint32_t*>(s_b + swz(j, nk) + nb);
      }
      const uint32_t a01 = __builtin_amdgcn_perm(r[1], r[0], 0x05010400u);
      const uint32_t b01 = __builtin_amdgcn_perm(r[1], r[0], 0x07030602u);
      const uint32_t a23 = __builtin_amdgcn_perm(r[3], r[2], 0x05010400u);
      const uint32_t b23 = __builtin_amdgcn_perm(r[3], r[2], 0x07030602u);
      col[0][g4] = __builtin_amdgcn_perm(a23, a01, 0x05040100u);
      col[1][g4] = __builtin_amdgcn_perm(a23, a01, 0x07060302u);
      col[2][g4] = __builtin_amdgcn_perm(b23, b01, 0x05040100u);
      col[3][g4] = __builtin_amdgcn_perm(b23, b01, 0x07060302u);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *reinterpret_cast<uint4*>(dst + frag::kslice_offset(n0 + i, j0, kQ)) =
          make_uint4(col[i][0], col[i][1], col[i][2], col[i][3]);
  }

  // ---- the causal 32x32 tiles of row blocks [jlo, jhi) (global tile numbers [jlo (jlo + 1) / 2,
  //      jhi (jhi + 1) / 2)), wave w taking the part's tiles w, w + 8, ...
  const int hl = lane >> 5, lr = lane & 31;
  const int tile_end = jhi * (jhi + 1) / 2;
  for (int tile = jlo * (jlo + 1) / 2 + wv; tile < tile_end; tile += kWaves) {
    int jt = 0, it = tile;
    while (it > jt) { it -= jt + 1; ++jt; }
    v4i a[4], bb[4];
#pragma unroll
    for (int ks = 0; ks < kN / 32; ++ks) {
      a[ks] = *reinterpret_cast<const v4i*>(s_c + swz(jt * 32 + lr, 2 * ks + hl));
      bb[ks] = *reinterpret_cast<const v4i*>(s_b + swz(it * 32 + lr, 2 * ks + hl));
    }
    if (it == 0) {
      // the C_q rows of block jt, in ChunkScan1 fragment order
      int8_t* cdst = cq_frag + cg * (size_t)kQ * kN;
      if (cq_perm) {
        // permuted kslice order: lane (j, h) holds n = 8 g + 4 h + [0, 4) at dword g; it has
        // n = 16 h + [0, 16): the lower half-wave keeps its dwords 0 and 2 and takes the upper
        // half's 0 and 2, the upper half keeps 1 and 3 and takes the lower half's 1 and 3
#pragma unroll
        for (int ks = 0; ks < kN / 32; ++ks) {
          const auto s01 = __builtin_amdgcn_permlane32_swap(a[ks][0], a[ks][1], false, false);
          const auto s23 = __builtin_amdgcn_permlane32_swap(a[ks][2], a[ks][3], false, false);
          *reinterpret_cast<uint4*>(cdst + ((size_t)jt * (kN / 32) + ks) * 1024 + lane * 16) =
              make_uint4(s01[0], s23[0], s01[1], s23[1]);
        }
      } else {
#pragma unroll
        for (int ks = 0; ks < kN / 32; ++ks)
          *reinterpret_cast<v4i*>(cdst + frag::kslice_offset(jt * 32 + lr, 32 * ks + 16 * hl,
                                                             kN)) = a[ks];
      }
    }
    // CB32^T: lane l holds target row j = 32 jt + l % 32 and, in register r, source token
    // i = 32 it + 8 (r / 4) + 4 (l / 32) + r % 4, so one requant multiplier serves the lane
    v16i acc = {};
#pragma unroll
    for (int ks = 0; ks < kN / 32; ++ks)
      acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(bb[ks], a[ks], acc, 0, 0, 0);
    const int j = jt * 32 + lr;
    const float m = s_m[j];
    uint32_t d[4];   // codes + 128 of i = 32 it + 8 g4 + 4 (l / 32) + [0, 4)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      uint32_t bits[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int ii = 8 * g4 + 4 * hl + e;
        const bool keep = it < jt || ii <= lr;
        bits[e] = keep ? requant_bits(acc[4 * g4 + e], m) : 0x4B400000u;   // 0x4B400000: code 0
      }
      d[g4] = pack_lo4(bits[0], bits[1], bits[2], bits[3]) ^ 0x80808080u;   // stored as q + 128
    }
    if (cbq_tap || cb32_tap) {   // row-major debug copies
      const size_t orow = cg * (size_t)kQ * kQ + (size_t)j * kQ + it * 32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ii = 8 * (r >> 2) + 4 * hl + (r & 3);
        const bool keep = it < jt || ii <= lr;
        if (cbq_tap) cbq_tap[orow + ii] = (int8_t)(((d[r >> 2] >> (8 * (r & 3))) & 0xffu) ^ 0x80u);
        if (cb32_tap) cb32_tap[orow + ii] = keep ? acc[r] : 0;
      }
    }
    // CB order wants i = 32 it + 8 (l / 32) + [0, 8) and 16 + that: the lower half-wave keeps
    // runs 0 and 2 and takes the upper half's runs 0 and 2, the upper half keeps runs 1 and 3
    // and takes the lower half's runs 1 and 3 (lanes l and l ^ 32 exchange one dword each)
    const auto s01 = __builtin_amdgcn_permlane32_swap(d[0], d[1], false, false);
    const auto s23 = __builtin_amdgcn_permlane32_swap(d[2], d[3], false, false);
    *reinterpret_cast<uint4*>(cbq_frag + cg * (size_t)frag::kCbChunkBytes +
                              (size_t)frag::cb_block(jt, it) * 1024 + lane * 16) =
        make_uint4(s01[0], s01[1], s23[0], s23[1]);
  }
}

}  // namespace

hipError_t launch_chunk_bmm(const LayerDims& d, const void* C, const void* B, int src_dtype,
                            const float* C_scale, int c_per_token, const float* B_scale,
                            const float* cb_scale, int8_t* cbq_frag, int8_t* cbq_tap,
                            int32_t* cb32_tap, int8_t* bqT_frag, int8_t* cq_frag, int cq_perm,
                            int* sync, int nsync, int* timeouts, hipStream_t st,
                            hipEvent_t ev_start, hipEvent_t ev_stop) {
  const int64_t ncg = (int64_t)d.batch * d.nchunks * d.ngroups;
  // parts per chunk-group: enough workgroups to reach every CU on small layers
  const int S = ncg <= 128 ? 4 : (ncg <= 256 ? 2 : 1);
  const int64_t nwork = ncg * S;
  if (nwork == 0) return hipSuccess;
#define SSDI8_BMM_ARGS(T)                                                                       \
  static_cast<const T*>(C), static_cast<const T*>(B), C_scale, c_per_token, B_scale, cb_scale,  \
      cbq_frag, cbq_tap, cb32_tap, bqT_frag, cq_frag, cq_perm, sync, nsync, timeouts, d.seqlen, \
      d.ngroups, d.nchunks, S
#define SSDI8_BMM_LAUNCH(T)                                                                     \
  do {                                                                                          \
    if (ev_start || ev_stop)                                                                    \
      hipExtLaunchKernelGGL(chunk_bmm_kernel<T>, dim3((unsigned)nwork), dim3(kThreads), 0, st, \
                            ev_start, ev_stop, 0, SSDI8_BMM_ARGS(T));                           \
    else                                                                                        \
      hipLaunchKernelGGL(chunk_bmm_kernel<T>, dim3((unsigned)nwork), dim3(kThreads), 0, st,    \
                         SSDI8_BMM_ARGS(T));                                                    \
  } while (0)
  if (src_dtype < 0) SSDI8_BMM_LAUNCH(int8_t);
  else if (src_dtype == 1) SSDI8_BMM_LAUNCH(_Float16);
  else SSDI8_BMM_LAUNCH(float);
#undef SSDI8_BMM_LAUNCH
#undef SSDI8_BMM_ARGS
  return hipGetLastError();
}

}  // namespace ssdi8
