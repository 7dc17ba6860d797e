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
// costs two fp32 products and no exp.  A diagonal block splits the same way about r_{J-1}
// (exp(cs_j - r_{J-1}) exp(r_{J-1} - cs_i)) when its span r_{J-1} - r_J is small enough for the
// second factor to stay finite; otherwise it evaluates exp per element.
//
// Work split: wave w owns the j-blocks {w, 7-w} (1+w + 8-w = 9 causal block pairs per wave).
// Strong decay removes work exactly: leading off-diagonal blocks whose fp16 weights all round to
// zero are not formed, and Scan1 is not run for a j-block whose factor exp(cs_j) is zero in fp32.
// x is staged once in LDS as x^T [p][i] (fp16, tokens contiguous = the Scan2 MFMA K-slice); the
// D skip term reads it back per token, and the fp16 output leaves through the same bytes as whole
// 128-byte rows.  C_q, P_in and CB_q arrive in MFMA fragment order (frag.hpp), so every operand
// load is one contiguous 1 KB run per wave.  Under 40 KB of LDS and at most 128 VGPRs per lane
// let four workgroups share a CU.
#include <hip/hip_ext.h>

#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

namespace ssdi8 {

namespace {

constexpr int kXTS = kQ * 2 + 16;   // bytes per channel row of x^T (fp16)
constexpr int kXQS = kQ + 16;       // bytes per channel row of X_q^T (int8, single pass)
static_assert(kP * kXTS >= kQ * kP * 2, "the fp16 output stage reuses the x^T bytes");
// A diagonal block whose decay span r_{J-1} - r_J stays below this bound forms its weights as
// (a_CB dt_i exp(-(cs_i - r_{J-1}))) * exp(cs_j - r_{J-1}) without overflow in fp32.
constexpr float kDiagSpan = 64.0f;
// Single pass: how many earlier chunks a chunk looks back over for a published entering state,
// and the status bits of a chunk's flag word (its Q(Decay) in the low 16 bits).
constexpr int kLook = 4;
constexpr uint32_t kFlagS = 1u << 16;   // the chunk-local S_q of the chunk is published
constexpr uint32_t kFlagP = 1u << 17;   // the state entering the next chunk is published

// Two adjacent channels of one token row, loaded raw and converted to fp16 for the MFMA.
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

// kMode: 0 the separate ChunkScan, 1 the single pass, 2 the single pass with speculative first
// loads (kSpec below).
template <typename XT, typename YT, int kMode>
__global__ __launch_bounds__(256, 4) void chunk_scan_kernel(
    const XT* __restrict__ x, const float* __restrict__ dt, const float* __restrict__ A,
    const int8_t* __restrict__ cq_frag, const float* __restrict__ C_scale, int c_per_token,
    int8_t* __restrict__ pin, const int8_t* __restrict__ cbq,
    const float* __restrict__ cb_scale, const float* __restrict__ state_scale,
    const float* __restrict__ Dv, const float* __restrict__ corr, int dt_softplus,
    YT* __restrict__ y, int32_t* __restrict__ y1_tap, int L, int H, int G, int nc,
    FusedState fs) {
  constexpr bool kFused = kMode != 0;
  constexpr bool kSpec = kMode == 2;
  // One LDS block with the small per-token tables first, so that their offsets fit the 16-bit
  // ds offset field (separate __shared__ arrays may be placed large-first).
  struct __attribute__((aligned(16))) Smem {
    // Column tables of the ChunkScan2 weights, interleaved as (w, -128 w) pairs so that an int8
    // weight q, converted as the unsigned byte q + 128, gives fl32(q w) = fma(q + 128, w, -128 w)
    // exactly (the fma forms (q + 128) w - 128 w = q w before its one rounding).
    union {
      float2 u[kQ];      // a_CB dt_i exp(r_I - cs_i)                  (off-diagonal blocks)
      float lut[kQ];     // single pass: LUT_state of ChunkState, read before u is built
    };
    float2 dg[kQ];       // a_CB dt_i exp(r_{I-1} - cs_i) if block I has a small span, else
                         // a_CB dt_i                                   (diagonal blocks)
    float csr[kQ];       // cs_i - r_{I-1} (r_{-1} = 0), fp32
    float R[8][8];       // exp(r_a - r_b), b <= a
    float umax[8];       // max |u_i| over block I (inf if one is NaN)
    int it0[8];          // single pass: the first ChunkScan2 block run by row block J
    float aS[kP];
    float cr[kP];
    double r[8];         // r_t: cs at the last token of block t
    double scan[kScanScratch];
    int misc[4];         // single pass: ticket, q_d, look-back anchor
    int lq[kLook];       // single pass: Q(Decay) of chunks c-1, c-2, ... (flag words' low half)
    // x^T [p][i] fp16: the ChunkScan2 MFMA operand and, for fp16 x, the D skip operand; then
    // the stage of the fp16 output (256 rows of 128 bytes).  16-byte aligned whatever the
    // tables before it add up to: its 128-bit accesses split when it is not (a look-back depth
    // that left it 4- or 8-byte aligned ran the single pass 34-55 % slower).
    alignas(16) uint8_t xT[kP * kXTS];
  };
  __shared__ Smem sm;
  float2* s_u = sm.u;
  float2* s_dg = sm.dg;
  float* s_csr = sm.csr;
  float (*s_R)[8] = sm.R;
  float* s_aS = sm.aS;
  float* s_cr = sm.cr;
  double* s_r = sm.r;
  double* s_scan = sm.scan;
  uint8_t* s_xT = sm.xT;

  const int t = threadIdx.x, lane = t & 63;
  const int wv = __builtin_amdgcn_readfirstlane(t >> 6);   // wave-uniform, so block loops are scalar
  int b, c, h;
  // x tile (thread: channel pair (p0, p0+1), tokens [32 jb, 32 jb + 32))
  const int pp = t & 31, jb = t >> 5, p0 = 2 * pp;
  // single pass: wave -> channel tile mt and state tiles ntb, ntb + 1; lane -> channel prow
  const int hf = lane >> 5, mt = wv & 1, ntb = (wv >> 1) * 2;
  const int prow = mt * 32 + (lane & 31);
  // ---- loads in the order they are needed (vector loads complete in issue order): dt and the
  //      per-channel tables first, so that the block scan and the tables wait for them alone
  //      while the x tile is still in flight.  The single pass also requests the X_q steps of
  //      this thread's channel pair and the steps of this lane's channel for the ChunkState
  //      requant (unconditional loads, so that none of the waits before them is a full drain).
  float dtv, aSv, crv, ax0 = 1.0f, ax1 = 1.0f, axs = 1.0f, asp = 1.0f, abq = 1.0f;
  auto item_loads = [&](int bb, int cc, int hh) {
    const int gg = __builtin_amdgcn_readfirstlane(hh / (H / G));
    const size_t t0 = (size_t)bb * L + (size_t)cc * kQ;
    dtv = dt[(t0 + t) * H + hh];
    aSv = t < kP ? state_scale[hh * kP + t] : 0.0f;
    crv = (t < kP && corr) ? corr[hh * kP + t] : 0.0f;
    if constexpr (kFused) {
      const int xo = fs.xs_per_head ? 0 : 1;
      ax0 = fs.xs_scale[xo * (hh * kP + p0) + (1 - xo) * hh];
      ax1 = fs.xs_scale[xo * (hh * kP + p0 + 1) + (1 - xo) * hh];
      axs = fs.xs_scale[xo * (hh * kP + prow) + (1 - xo) * hh];
      asp = state_scale[hh * kP + prow];
      abq = fs.B_scale[gg];
    }
  };
  if constexpr (kFused) {
    // Work items in ticket order.  The sequences (b, h) are split into K blocks of consecutive
    // sequences, one per class; class x hands out its items chunk-major from its own counter, so
    // the item a workgroup waits for (same sequence, previous chunk) holds an earlier ticket of
    // the same counter and is running or done.  A workgroup draws from class blockIdx % K and,
    // once that class is exhausted, from the next ones; the grid has as many workgroups as
    // items, so every item is drawn.  K (a multiple of 8) is chosen so that each class holds as
    // many items as workgroups start on it, and each counter sits on its own cache line: the
    // atomics of a launch spread over K lines instead of queueing on one.  With round-robin
    // dispatch over the 8 XCDs, class x runs on XCD x % 8, and the K / 8 classes of one XCD take
    // consecutive sequence blocks, so that the heads of one batch element (which share the
    // chunk's B_q^T, C_q and CB_q) meet in as few L2 caches as possible.
    const int nbh = fs.nbh, K = fs.nclass;
    const int q = nbh / K, r = nbh - q * K;
    auto decode = [&](int it, int& bb, int& cc, int& hh) {
      cc = it / nbh;
      const int bh = it - cc * nbh;
      bb = bh / H;
      hh = bh - bb * H;
    };
    // kSpec (grids of about one round of workgroups, where every item's first loads wait in
    // full): the item drawn when tickets follow dispatch order, the (blockIdx / K)-th ticket of
    // class blockIdx % K, has its loads requested while the ticket is drawn (after the ticket's
    // atomic, which they must not delay), and they are requested again only if it differs
    int pred = -1, tk0 = 0;
    if constexpr (kSpec) {
      const int x = (int)(blockIdx.x & (K - 1));
      const int sb = (x & 7) * (K >> 3) + (x >> 3);
      const int chains = q + (sb < r ? 1 : 0);
      const int tk = (int)(blockIdx.x / K);
      if (chains > 0 && tk < chains * nc) {
        const int cc = tk / chains;
        pred = cc * nbh + sb * q + (sb < r ? sb : r) + (tk - cc * chains);
      }
      pred = __builtin_amdgcn_readfirstlane(pred);
      if (t == 0) tk0 = atomicAdd(fs.sync + x * kSyncLine, 1);
      int pb, pc, ph;
      decode(pred < 0 ? 0 : pred, pb, pc, ph);
      item_loads(pb, pc, ph);
    }
    if (t == 0) {
      int item = -1;
      for (int k = 0; k < K && item < 0; ++k) {
        const int x = (int)((blockIdx.x + k) & (K - 1));
        const int sb = (x & 7) * (K >> 3) + (x >> 3);   // sequence block of class x
        const int chains = q + (sb < r ? 1 : 0);
        if (chains <= 0) continue;
        const int tk = (kSpec && k == 0) ? tk0 : atomicAdd(fs.sync + x * kSyncLine, 1);
        if (tk < chains * nc) {
          const int cc = tk / chains;
          item = cc * nbh + sb * q + (sb < r ? sb : r) + (tk - cc * chains);
        }
      }
      sm.misc[0] = item;
    }
    __syncthreads();
    const int item = __builtin_amdgcn_readfirstlane(sm.misc[0]);
    if (item < 0) return;   // every item drawn (only with an uncleared counter)
    decode(item, b, c, h);
    if (!kSpec || item != pred) item_loads(b, c, h);
  } else {
    const int w = xcd_remap(blockIdx.x, gridDim.x);
    h = w % H;
    const int bc = w / H;
    c = bc % nc;
    b = bc / nc;
    item_loads(b, c, h);
  }
  // wave-uniform (the division is done on the vector unit), so that the per-group steps are
  // scalar loads and none of them drains the vector loads in flight
  const int g = __builtin_amdgcn_readfirstlane(h / (H / G));
  const size_t tok0 = (size_t)b * L + (size_t)c * kQ;
  const size_t HP = (size_t)H * kP;
  const float aCB = cb_scale[g];
  typename Pair<XT>::raw xr[32];
  {
    const __amdgpu_buffer_rsrc_t xrs = buffer_rsrc(x + tok0 * HP + (size_t)h * kP);
    const uint32_t xo = (uint32_t)((jb * 32 * HP + p0) * sizeof(XT));
    // x and y are touched once: streamed (non-temporal) when the layer's x and y exceed the
    // Infinity Cache, so that they do not displace the tiles every head of a chunk reuses
    if (fs.stream) {
#pragma unroll
      for (int r = 0; r < 32; ++r)
        xr[r] = Pair<XT>::template load<kPolicyNT>(xrs, xo, (uint32_t)(r * HP * sizeof(XT)));
    } else {
#pragma unroll
      for (int r = 0; r < 32; ++r) xr[r] = Pair<XT>::load(xrs, xo, (uint32_t)(r * HP * sizeof(XT)));
    }
  }
  // ---- ChunkCumsum (fp64 sums; the factors derived from it only need fp32 accuracy here).
  //      dt is the fp64 softplus rounded once to fp32, as in ChunkState: one dt per token for
  //      the whole layer (and X_scaled of the single pass needs exactly that value)
  if (dt_softplus) dtv = softplus_f32(dtv);
  const float dA = dtv * A[h];
  const double cs = block_scan_f64_256(dA, s_scan, sm.lut);
  if ((t & 31) == 31) s_r[t >> 5] = cs;
  if (t < kP) {
    s_aS[t] = aSv;
    s_cr[t] = crv;
  }
  __syncthreads();
  // ChunkScan2's tables (the single pass builds them after ChunkState: u shares LDS with LUT)
  auto scan_tables = [&]() {
    const int blk = t >> 5;
    const double rprev = blk ? s_r[blk - 1] : 0.0;
    const float dtcb = aCB * dtv;
    const float u = dtcb * expf((float)(s_r[blk] - cs));
    s_u[t] = make_float2(u, -128.0f * u);
    float um = u == u ? __builtin_fabsf(u) : __builtin_inff();
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) um = __builtin_fmaxf(um, __shfl_xor(um, o));
    if ((t & 31) == 0) sm.umax[blk] = um;
    const float csr = (float)(cs - rprev);
    s_csr[t] = csr;
    // the same test as the diagonal block's (on its last token's csr)
    const bool small_span = (float)(s_r[blk] - rprev) >= -kDiagSpan;
    const float dg = small_span ? dtcb * expf(__builtin_fminf(-csr, kDiagSpan)) : dtcb;
    s_dg[t] = make_float2(dg, -128.0f * dg);
    if (t < 64) {
      const int ra = t >> 3, rb = t & 7;
      s_R[ra][rb] = (rb <= ra) ? expf((float)(s_r[ra] - s_r[rb])) : 0.0f;
    }
  };
  if constexpr (!kFused) scan_tables();
  if constexpr (kFused) {
    // ChunkState's table and Q(Decay), with its exact arithmetic (Eq. 4, Eq. 9)
    const double last = s_r[7];
    sm.lut[t] = dtv * (float)exp(last - cs);
    if (t == 0) sm.misc[1] = (int)rint(exp(last) * (double)(1 << fs.shift));
  }
  // ---- x^T [p][i] (fp16) in LDS
  auto stage_xT = [&]() {
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
  };
  if constexpr (!kFused) {
    stage_xT();
  } else {
    // single pass: X_q^T [p][j] (int8, Eq. 7) first, in the bytes x^T takes later: each x
    // element is quantized once, by the thread that loaded it, with ChunkState's arithmetic
    __syncthreads();   // LUT_state complete
    const float inv0 = 1.0f / ax0, inv1 = 1.0f / ax1;
    uint32_t w0[8], w1[8];
#pragma unroll
    for (int r4 = 0; r4 < 8; ++r4) {
      uint32_t qa[4], qb[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * r4 + i;
        const float lut = sm.lut[jb * 32 + r];
        // fl32(lut x) as one mixed-precision fma with +0 (only a zero product's sign can
        // differ, and it quantizes to 0 either way)
        qa[i] = quant_bits(
            __builtin_fmaf(lut, (float)__builtin_bit_cast(_Float16, Pair<XT>::lo(xr[r])), 0.0f),
            inv0);
        qb[i] = quant_bits(
            __builtin_fmaf(lut, (float)__builtin_bit_cast(_Float16, Pair<XT>::hi(xr[r])), 0.0f),
            inv1);
      }
      w0[r4] = pack_lo4(qa[0], qa[1], qa[2], qa[3]);
      w1[r4] = pack_lo4(qb[0], qb[1], qb[2], qb[3]);
    }
    uint8_t* q0 = s_xT + p0 * kXQS + jb * 32;
    *reinterpret_cast<uint4*>(q0) = make_uint4(w0[0], w0[1], w0[2], w0[3]);
    *reinterpret_cast<uint4*>(q0 + 16) = make_uint4(w0[4], w0[5], w0[6], w0[7]);
    *reinterpret_cast<uint4*>(q0 + kXQS) = make_uint4(w1[0], w1[1], w1[2], w1[3]);
    *reinterpret_cast<uint4*>(q0 + kXQS + 16) = make_uint4(w1[4], w1[5], w1[6], w1[7]);
  }
  __syncthreads();

  uint32_t sq[2][4];   // S_q of the two tiles, byte r of word r / 4 = MFMA result row r
  if constexpr (kFused) {
    // ---- ChunkState (Eq. 7-8), transposed: S32^T = B_q^T X_q with the X_q^T fragments staged
    //      above.  Lane -> channel p = 32 mt + l % 32 and, per tile, the 16 state rows n of the
    //      permuted kslice order (frag.hpp), which is where the MFMA leaves them.
    const float msp = (float)(((double)axs * (double)abq) / (double)asp);
    {
      const __amdgpu_buffer_rsrc_t brs =
          buffer_rsrc(fs.bqT + (((size_t)b * nc + c) * G + g) * (size_t)kN * kQ);
      const uint32_t l16 = lane * 16;
      v16i s0 = {}, s1 = {};
      const uint8_t* arow = s_xT + prow * kXQS + 16 * hf;
#pragma unroll
      for (int ks = 0; ks < kQ / 32; ++ks) {
        const v4i bf0 = __builtin_bit_cast(
            v4i, buf_load16(brs, l16, (uint32_t)((ntb * (kQ / 32) + ks) * 1024)));
        const v4i bf1 = __builtin_bit_cast(
            v4i, buf_load16(brs, l16, (uint32_t)(((ntb + 1) * (kQ / 32) + ks) * 1024)));
        const v4i a = *reinterpret_cast<const v4i*>(arow + ks * 32);
        s0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(bf0, a, s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(bf1, a, s1, 0, 0, 0);
      }
      // S_q = requant(S32, m_S[p]) (Eq. 8), one multiplier per lane
#pragma unroll
      for (int w4 = 0; w4 < 4; ++w4) {
        sq[0][w4] = pack_lo4(requant_bits(s0[4 * w4], msp), requant_bits(s0[4 * w4 + 1], msp),
                             requant_bits(s0[4 * w4 + 2], msp), requant_bits(s0[4 * w4 + 3], msp));
        sq[1][w4] = pack_lo4(requant_bits(s1[4 * w4], msp), requant_bits(s1[4 * w4 + 1], msp),
                             requant_bits(s1[4 * w4 + 2], msp), requant_bits(s1[4 * w4 + 3], msp));
      }
    }
    // X_q^T and LUT_state no longer read: x^T and ChunkScan2's tables (u over LUT) take their
    // bytes
    __syncthreads();
    stage_xT();
    scan_tables();
    __syncthreads();
  }

  // The first off-diagonal ChunkScan2 block that row block jt runs: leading blocks whose every
  // fp16 weight rounds to zero are skipped (see the j-block).  jt itself when all are skipped.
  auto first_block = [&](int jt) {
    if (jt <= 0) return 0;
    const float4 ua = *reinterpret_cast<const float4*>(sm.umax);
    const float4 ub = *reinterpret_cast<const float4*>(sm.umax + 4);
    const float4 ra = *reinterpret_cast<const float4*>(s_R[jt - 1]);
    const float4 rb = *reinterpret_cast<const float4*>(s_R[jt - 1] + 4);
    const float um[8] = {ua.x, ua.y, ua.z, ua.w, ub.x, ub.y, ub.z, ub.w};
    const float rr[8] = {ra.x, ra.y, ra.z, ra.w, rb.x, rb.y, rb.z, rb.w};
    uint32_t live = 1u << jt;   // the diagonal block always runs
#pragma unroll
    for (int k = 0; k < 7; ++k)
      if (!(um[k] * rr[k] < 0x1p-33f)) live |= 1u << k;
    return (int)__builtin_ctz(live);
  };

  // ---- single pass, StatePassing (Eq. 9) for this chunk.  P_in[c], the state entering the
  //      chunk, comes from the chunks before it in its sequence.  The flag word of chunk m holds
  //      its Q(Decay) in the low 16 bits and two status bits: kFlagS (its chunk-local S_q is in
  //      the sq slot of (b, m, h)) and kFlagP (P_in[m+1] is in the pin slot of (b, m+1, h)).
  //      With kFlagP at chunk c-1-l (l < kLook) and kFlagS on every chunk in between,
  //      P_in[c] = Eq. 9 applied to P_in[c-l] over the S_q of chunks c-l, ..., c-1 in chunk order:
  //      the same recurrence, hence the same integers as a chain of hand-offs from chunk to
  //      chunk, without waiting for each of them.  A chunk that finds no such anchor at its first
  //      look publishes its own S_q (so that later chunks can look past it), then polls until it
  //      does; every chunk then publishes P_in[c+1] (a chunk with Q(Decay) = 0 does so before
  //      its first look, see below).  Only earlier chunks of the same sequence are waited for;
  //      they hold earlier tickets of the same counter, so each is running or done, publishes
  //      its S_q or its P_in[m+1] before it waits, and chunk 0 waits for nothing.  Waits are
  //      bounded: one that runs out is counted (sync[kSyncWait] and the caller's counter) and the
  //      kernel still finishes.  Each lane updates its own 32 state bytes in registers; payloads
  //      are written and read at the agent's coherence point (sc1) and are complete before
  //      their flag is set.
  auto hand_off = [&]() {
    // the first ChunkScan2 block of each row block, for the j-blocks after the hand-off's last
    // barrier (the tables are complete)
    if (wv == 0 && lane < 8) sm.it0[lane] = first_block(lane);
    constexpr size_t kSlab = (size_t)kP * kN;
    constexpr int kPolicySc1 = 16;
    const int bh = b * H + h;
    int* flags = fs.sync + kSyncFlags + (size_t)bh * nc;   // flag of chunk m at flags[m]
    const int qd = __builtin_amdgcn_readfirstlane(sm.misc[1]);
    auto slab_of = [&](int8_t* base, int cc) {
      return base + (((size_t)b * nc + cc) * H + h) * kSlab;
    };
    // this lane's 16-byte slices of the two state tiles of a slab
    const uint32_t off0 = (uint32_t)((mt * (kN / 32) + ntb) * 1024 + lane * 16);
    const uint32_t off1 = off0 + 1024;
    auto ld_sc1 = [&](const int8_t* slab, uint32_t off) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(buffer_rsrc(slab), (int)off, 0,
                                                           kPolicySc1);
      return make_uint4(v[0], v[1], v[2], v[3]);
    };
    auto st_sc1 = [&](uint4 d, int8_t* slab, uint32_t off) {
      typedef uint32_t u32x4 __attribute__((vector_size(16)));
      const u32x4 v = {d.x, d.y, d.z, d.w};
      __builtin_amdgcn_raw_buffer_store_b128(v, buffer_rsrc(slab), (int)off, 0, kPolicySc1);
    };
    // Eq. 9 on the 32 bytes of a lane: state st, chunk-local s, Q(Decay) q (packed 16-bit
    // arithmetic for shifts up to 8 and 0 <= q <= 2^shift, where it is exact; 32-bit
    // otherwise, e.g. for a decay above 1 from inputs outside the method's domain)
    auto step = [&](uint4 st, uint4 sl, int q) {
      const uint32_t a[4] = {st.x, st.y, st.z, st.w}, sv[4] = {sl.x, sl.y, sl.z, sl.w};
      uint32_t o[4];
      if (fs.shift <= 8 && q >= 0 && q <= (1 << fs.shift)) {
        const s16x2 q2 = {(short)q, (short)q}, r2 = {(short)fs.radd, (short)fs.radd};
        const s16x2 k2 = {(short)fs.shift, (short)fs.shift};
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) o[g4] = pass_step4_pk16(a[g4], sv[g4], q2, r2, k2);
      } else {
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          int v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            v[e] = pass_step(sext8(a[g4], e), sext8(sv[g4], e), q, fs.shift, fs.radd);
          o[g4] = pack4_i8(v[0], v[1], v[2], v[3]);
        }
      }
      return make_uint4(o[0], o[1], o[2], o[3]);
    };
    // wave 0: the flags of chunks c-1-lane (lane < kLook); the nearest anchor lane l, or -1
    auto look = [&](uint32_t* fout) {
      const int m = c - 1 - lane;
      uint32_t f = 0;
      if (lane < kLook && m >= 0)
        f = (uint32_t)__hip_atomic_load(flags + m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      *fout = f;
      const uint64_t mp = __ballot((f & kFlagP) != 0);
      const uint64_t ma = __ballot((f & (kFlagS | kFlagP)) != 0);
      const int lp = mp ? (int)__builtin_ctzll(mp) : 64;
      const int la = (int)__builtin_ctzll(~ma);   // lanes >= kLook never hold a status
      return (lp < kLook && la >= lp) ? lp : -1;
    };
    const uint4 sq0 = make_uint4(sq[0][0], sq[0][1], sq[0][2], sq[0][3]);
    const uint4 sq1 = make_uint4(sq[1][0], sq[1][1], sq[1][2], sq[1][3]);
    // With Q(Decay) = 0, Eq. 9 gives P_in[c+1] = clamp(S_q[c] + (r >> k)) whatever P_in[c] is:
    // such a chunk publishes P_in[c+1] before it obtains P_in[c], so that its successor finds
    // an anchor at once (the same integers; its S_q is then never needed by later chunks)
    const bool early = qd == 0 && c + 1 < nc;
    if (early) {
      // r < 2^k (r = 2^(k-1) or 0) makes it S_q[c] itself (codes within +-127)
      const bool same = (fs.radd >> fs.shift) == 0;
      const uint4 z = make_uint4(0u, 0u, 0u, 0u);
      int8_t* slab = slab_of(pin, c + 1);
      st_sc1(same ? sq0 : step(z, sq0, 0), slab, off0);
      st_sc1(same ? sq1 : step(z, sq1, 0), slab, off1);
    }
    // its flag, once every wave's stores are complete: for c > 0 together with the first look,
    // whose flag loads are in flight meanwhile (one wait and one barrier for both)
    auto publish_early = [&]() {
      if (t == 0)
        __hip_atomic_store(flags + c, (int)kFlagP, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    uint4 p0 = make_uint4(0u, 0u, 0u, 0u), p1 = p0;   // P_in[c]
    // an early chunk whose predecessor had published P_in[c] uses it only in ChunkScan1, which
    // loads it itself: no state loads, no stores after the look, so no closing barrier
    bool quiet = false;
    if (c == 0) {
      if (early) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        publish_early();
      }
      // the initial state (row-major; 0 without one), also ChunkScan1's entering state of chunk 0
      uint32_t w[2][4];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        // row-major (p, n) of this lane's byte 4 g + e: p = prow, n = 32 (ntb + i) + 8 g + 4 hf + e
        const size_t rbase = (size_t)bh * kSlab + (size_t)prow * kN + 32 * (ntb + i) + 4 * hf;
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4)
          w[i][g4] = fs.init ? *reinterpret_cast<const uint32_t*>(fs.init + rbase + 8 * g4) : 0u;
      }
      p0 = make_uint4(w[0][0], w[0][1], w[0][2], w[0][3]);
      p1 = make_uint4(w[1][0], w[1][1], w[1][2], w[1][3]);
      int8_t* slab = slab_of(pin, 0);
      *reinterpret_cast<uint4*>(slab + off0) = p0;
      *reinterpret_cast<uint4*>(slab + off1) = p1;
    } else {
      if (wv == 0) {
        uint32_t f;
        const int l = look(&f);
        if (lane == 0) sm.misc[2] = l;
        if (lane < kLook) sm.lq[lane] = (int)(f & 0xffffu);
      }
      if (early) __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      if (early) publish_early();
      int l = __builtin_amdgcn_readfirstlane(sm.misc[2]);
      if (l < 0) {
        // publish S_q[c] for the chunks after this one (unless P_in[c+1] already is), then wait
        // for an anchor
        if (!early) {
          int8_t* sslab = slab_of(fs.sq, c);
          st_sc1(sq0, sslab, off0);
          st_sc1(sq1, sslab, off1);
          __builtin_amdgcn_s_waitcnt(0);
          __syncthreads();
        }
        if (wv == 0) {
          if (lane == 0 && !early)
            __hip_atomic_store(flags + c, (int)(kFlagS | (uint32_t)qd), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
          uint32_t f = 0;
          int found = -1;
          for (int it = 0; it < fs.spin_limit && found < 0; ++it) {
            __builtin_amdgcn_s_sleep(2);
            found = look(&f);
          }
          if (found < 0) {
            if (lane == 0) {
              atomicAdd(fs.sync + kSyncWait, 1);
              if (fs.timeouts) atomicAdd(fs.timeouts, 1);
            }
            found = 0;
          }
          if (lane == 0) sm.misc[2] = found;
          if (lane < kLook) sm.lq[lane] = (int)(f & 0xffffu);
        }
        __syncthreads();
        l = __builtin_amdgcn_readfirstlane(sm.misc[2]);
      }
      quiet = early && l == 0;
      // P_in[c-l] (published by the anchor chunk c-1-l) and the S_q of chunks c-l .. c-1, all
      // loads in flight together
      if (!quiet) {
        const int8_t* pslab = slab_of(pin, c - l);
        p0 = ld_sc1(pslab, off0);
        p1 = ld_sc1(pslab, off1);
        uint4 s0[kLook - 1], s1[kLook - 1];
#pragma unroll
        for (int k = 0; k < kLook - 1; ++k) {
          if (k < l) {
            const int8_t* sslab = slab_of(fs.sq, c - l + k);
            s0[k] = ld_sc1(sslab, off0);
            s1[k] = ld_sc1(sslab, off1);
          }
        }
#pragma unroll
        for (int k = 0; k < kLook - 1; ++k) {
          if (k < l) {
            const int qk = sm.lq[l - 1 - k];   // Q(Decay) of chunk c - l + k
            p0 = step(p0, s0[k], qk);
            p1 = step(p1, s1[k], qk);
          }
        }
        if (l > 0) {
          // ChunkScan1 reads the entering state from the pin slot of this chunk
          int8_t* slab = slab_of(pin, c);
          st_sc1(p0, slab, off0);
          st_sc1(p1, slab, off1);
        }
      }
    }
    // P_in[c+1] = clamp(S_q[c] + ((q_d P_in[c] + r) >> k))
    if (c + 1 < nc) {
      if (!early) {
        int8_t* slab = slab_of(pin, c + 1);
        st_sc1(step(p0, sq0, qd), slab, off0);
        st_sc1(step(p1, sq1, qd), slab, off1);
      }
    } else {
      const uint4 n0 = step(p0, sq0, qd), n1 = step(p1, sq1, qd);
      const float a = s_aS[prow];   // state_scale[h, prow], staged in LDS at the start
      const uint32_t nw[2][4] = {{n0.x, n0.y, n0.z, n0.w}, {n1.x, n1.y, n1.z, n1.w}};
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const size_t rbase = (size_t)bh * kSlab + (size_t)prow * kN + 32 * (ntb + i) + 4 * hf;
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          if (fs.final_q) *reinterpret_cast<uint32_t*>(fs.final_q + rbase + 8 * g4) = nw[i][g4];
          if (fs.final_state)
            *reinterpret_cast<float4*>(fs.final_state + rbase + 8 * g4) =
                make_float4((float)sext8(nw[i][g4], 0) * a, (float)sext8(nw[i][g4], 1) * a,
                            (float)sext8(nw[i][g4], 2) * a, (float)sext8(nw[i][g4], 3) * a);
        }
      }
    }
    if (!quiet) {
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    }
    if (t == 0 && c + 1 < nc && !early)
      __hip_atomic_store(flags + c, (int)(kFlagP | (uint32_t)qd), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  };

  // Both products are formed transposed (MFMA rows = channels p, columns = tokens j), so each
  // lane owns one token row j and runs of 4 consecutive channels: the epilogue needs one row
  // factor per lane and moves 8-byte vectors.  Lane l: j = 32 jt + (l % 32); accumulator
  // register r holds channel p = 32 pt + 8 (r / 4) + 4 (l / 32) + r % 4.
  // operand fragments (frag.hpp): 1 KB per fragment, this lane's 16 bytes at lane * 16
  const int pc = lane & 31, half = lane >> 5;
  const size_t cg = ((size_t)b * nc + c) * G + g;
  const uint32_t lane16 = lane * 16;
  const __amdgpu_buffer_rsrc_t prs =
      buffer_rsrc(pin + (((size_t)b * nc + c) * H + h) * (size_t)kP * kN);
  const __amdgpu_buffer_rsrc_t cbrs = buffer_rsrc(cbq + cg * (size_t)frag::kCbChunkBytes);
  const __amdgpu_buffer_rsrc_t cqrs = buffer_rsrc(cq_frag + cg * (size_t)kQ * kN);
  const float Dh = Dv ? Dv[h] : 0.0f;
  // packed fp16 output of the two j-blocks (8 runs of 4 channels each), staged after the loop
  uint2 y_first[8], y_second[8];

  // One j-block of 32 tokens: Scan1, Scan2 and the epilogue; fp16 output packed into yo.
  auto jblock = [&](int jt, uint2 (&yo)[8]) {
    // keeps the per-channel epilogue tables of the two calls from being loaded once and held
    // across both (64 registers), and their addresses from being computed ahead of the call
    asm volatile("" : "+s"(jt) :: "memory");
    const int jrow = jt * 32 + pc;
    // the C step of this row, for the epilogue (requested first: its wait then drains nothing)
    const float ac = c_per_token ? C_scale[(tok0 + jrow) * G + g] : C_scale[g];
    const float csrj = s_csr[jrow];
    const float ej = __expf(csrj);                         // exp(cs_j - r_{J-1}), in (0, 1]
    const size_t orow = (tok0 + jrow) * HP + (size_t)h * kP;
    // -- the Scan2 accumulators start from D x + corr[p] (the skip and correction terms)
    v16f yd0, yd1;
#pragma unroll
    for (int pt = 0; pt < 2; ++pt) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int pb = pt * 32 + 8 * g4 + 4 * half;
        const float4 cr4 = *reinterpret_cast<const float4*>(s_cr + pb);
        const float crv[4] = {cr4.x, cr4.y, cr4.z, cr4.w};
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
          const float v0 = __builtin_fmaf(Dh, xv[q], crv[q]);
          if (pt) yd1[4 * g4 + q] = v0;
          else yd0[4 * g4 + q] = v0;
        }
      }
    }
    v4i a[4], b0[4], b1[4];   // ChunkScan1 operands
    // -- Scan2: y_diag^T = x^T . W^T, fp16 MFMA over the causal source tokens i; CB_q of
    //    block it+1 is prefetched while block it is built
    {
      const uint32_t cbrow = frag::cb_block(jt, 0) * 1024;   // blocks (jt, it)
      const bool diag_fast =
          __builtin_amdgcn_readfirstlane((int)(s_csr[jt * 32 + 31] >= -kDiagSpan)) != 0;
      // Leading off-diagonal blocks whose every weight rounds to an fp16 zero are skipped (the
      // decay across the blocks between them and this row block has removed them): a weight of
      // block it is q u_i e_j R[jt-1][it] with |q| <= 127 and e_j <= 1, below 127 2^-33 < 2^-26
      // when max |u_i| R < 2^-33, and such a value rounds to zero.  it0 = the first block run.
      int it0 = 0;
      if constexpr (kFused) {
        it0 = __builtin_amdgcn_readfirstlane(sm.it0[jt]);   // formed by the hand-off
      } else if (jt > 0) {
        it0 = __builtin_amdgcn_readfirstlane(first_block(jt));
      }
      // W^T fragment of a 32x32 block (8 weights of this lane's token row per K-slice, as fp16)
      // times the x^T fragments of both channel tiles
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
      // int8 weight e of a K-slice as the unsigned byte q + 128
      auto qbyte = [](uint32_t ub0, uint32_t ub1, int e) {
        return (float)(((e < 4 ? ub0 : ub1) >> (8 * (e & 3))) & 0xffu);
      };
      // CB_q fragments in a ring of three register sets: block it is built while blocks it+1 and
      // it+2 are in flight.  The off-diagonal steps are written out so that every slot stays a
      // fixed register set (a copy between slots would wait for the load in flight), and every
      // load is unconditional, its block index clamped to the row's last block jt (a branch
      // around a load makes the wait after it a full drain).
      auto blk = [&](int it) { return cbrow + (it < jt ? it : jt) * 1024; };
      uint4 r0 = buf_load16(cbrs, lane16, blk(it0));
      uint4 r1 = buf_load16(cbrs, lane16, blk(it0 + 1));
      uint4 r2;
      // off-diagonal block it < jt from slot cur; block min(it + 2, jt) into dst
      auto off_block = [&](const int it, const uint4& cur, uint4& dst) {
        dst = buf_load16(cbrs, lane16, blk(it + 2));
        // keep the prefetch at the top of the body
        __builtin_amdgcn_sched_barrier(0);
        // row factor: exp(cs_j - r_{J-1}) exp(r_{J-1} - r_I)
        const float vj = ej * s_R[jt - 1][it];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const int i0 = it * 32 + ks * 16 + 8 * half;
          const uint32_t ub0 = (ks ? cur.z : cur.x);
          const uint32_t ub1 = (ks ? cur.w : cur.y);
          float wv[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float2 uu = s_u[i0 + e];
            wv[e] = __builtin_fmaf(qbyte(ub0, ub1, e), uu.x, uu.y) * vj;
          }
          mfma_block(wv, i0);
        }
      };
      // block it0 + k sits in slot k % 3
      const int nb = jt - it0;
      if (nb > 0) {
        off_block(it0, r0, r2);
        if (nb > 1) {
          off_block(it0 + 1, r1, r0);
          if (nb > 2) {
            off_block(it0 + 2, r2, r1);
            if (nb > 3) {
              off_block(it0 + 3, r0, r2);
              if (nb > 4) {
                off_block(it0 + 4, r1, r0);
                if (nb > 5) {
                  off_block(it0 + 5, r2, r1);
                  if (nb > 6) off_block(it0 + 6, r0, r2);
                }
              }
            }
          }
        }
      }
      const int js = nb % 3;
      const uint4 cur = js == 0 ? r0 : (js == 1 ? r1 : r2);
      // the C_q fragments of ChunkScan1, in flight during the diagonal block
      {
        const uint32_t crow = jt * (kN / 32) * 1024;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
          a[ks] = __builtin_bit_cast(v4i, buf_load16(cqrs, lane16, crow + 1024 * ks));
        __builtin_amdgcn_sched_barrier(0);
      }
      // diagonal block it = jt: its entries i > j hold the code of zero, whose weight
      // fma(128, d, -128 d) is exactly +0, so no mask is needed
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int i0 = jt * 32 + ks * 16 + 8 * half;
        const uint32_t ub0 = (ks ? cur.z : cur.x);
        const uint32_t ub1 = (ks ? cur.w : cur.y);
        float wv[8];
        if (diag_fast) {
          // small span: exp(cs_j - cs_i) = exp(cs_j - r_{J-1}) exp(r_{J-1} - cs_i)
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float2 dd = s_dg[i0 + e];
            wv[e] = __builtin_fmaf(qbyte(ub0, ub1, e), dd.x, dd.y) * ej;
          }
        } else {
          // exp per element; the clamp keeps the (zero-weight) entries i > j finite
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float2 dd = s_dg[i0 + e];
            const float ex = __expf(__builtin_fminf(csrj - s_csr[i0 + e], 0.0f));
            wv[e] = __builtin_fmaf(qbyte(ub0, ub1, e), dd.x, dd.y) * ex;
          }
        }
        mfma_block(wv, i0);
      }
    }
    // -- Scan1: Y1^T = P_in . C_q^T, int8 MFMA over n.  Its term is Y1 a_C exp(cs_j) a_S[p];
    //    when exp(r_{J-1}) is zero in fp32 every factor exp(cs_j) of the block is a zero
    //    product and Y1 is not needed (unless it is tapped)
    const float er = jt ? __expf((float)s_r[jt - 1]) : 1.0f;
    const bool tap_y1 = !kFused && y1_tap;   // the single pass has no Y1 tap
    const bool need_y1 = tap_y1 || __builtin_amdgcn_readfirstlane((int)(er != 0.0f)) != 0;
    v16i yi0 = {}, yi1 = {};
    if (need_y1) {
      // the P_in fragments are the same for both j-blocks; an opaque offset makes each call
      // load them again (from L2) instead of holding 32 registers across the other block
      uint32_t lofs = lane16;
      asm volatile("" : "+v"(lofs));
      constexpr uint32_t p1row = (kN / 32) * 1024;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        b0[ks] = __builtin_bit_cast(v4i, buf_load16(prs, lofs, 1024 * ks));
        b1[ks] = __builtin_bit_cast(v4i, buf_load16(prs, lofs, p1row + 1024 * ks));
      }
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        yi0 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b0[ks], a[ks], yi0, 0, 0, 0);
        yi1 = __builtin_amdgcn_mfma_i32_32x32x32_i8(b1[ks], a[ks], yi1, 0, 0, 0);
      }
    }
    // -- epilogue of token row jrow: y = Y1 a_C exp(cs_j) a_S[p] + (y_diag + D x + corr[p])
    // a_C(j) exp(cs_j) = a_C(j) exp(cs_j - r_{J-1}) exp(r_{J-1})
    const float eo = ac * ej * er;
#pragma unroll
    for (int pt = 0; pt < 2; ++pt) {
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int pb = pt * 32 + 8 * g4 + 4 * half;
        const float4 as4 = *reinterpret_cast<const float4*>(s_aS + pb);
        const float asv[4] = {as4.x, as4.y, as4.z, as4.w};
        float v[4];
        int yi[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r = 4 * g4 + q;
          yi[q] = pt ? yi1[r] : yi0[r];
          const float yd = pt ? yd1[r] : yd0[r];
          v[q] = __builtin_fmaf((float)yi[q] * eo, asv[q], yd);
        }
        if (tap_y1)
          *reinterpret_cast<int4*>(y1_tap + orow + pb) = make_int4(yi[0], yi[1], yi[2], yi[3]);
        if constexpr (sizeof(YT) == 4) {
          *reinterpret_cast<float4*>(y + orow + pb) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          typedef float f2_t __attribute__((ext_vector_type(2)));
          typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
          const h2_t h01 = __builtin_convertvector((f2_t){v[0], v[1]}, h2_t);
          const h2_t h23 = __builtin_convertvector((f2_t){v[2], v[3]}, h2_t);
          uint2 o = make_uint2(__builtin_bit_cast(uint32_t, h01), __builtin_bit_cast(uint32_t, h23));
          // pinned here: otherwise the arithmetic sinks to the stage writes after the other
          // j-block and keeps this block's accumulators and tables alive across it
          asm volatile("" : "+v"(o.x), "+v"(o.y));
          yo[4 * pt + g4] = o;
        }
      }
    }
  };
  if constexpr (kFused) hand_off();
  jblock(wv, y_first);
  jblock(7 - wv, y_second);

  if constexpr (sizeof(YT) == 2) {
    // fp16 output leaves through LDS as whole 128-byte token rows.  The stage reuses the x^T
    // bytes once every wave is done with them: row j at 128 j, its 16-byte column chunk k at
    // slot k ^ (j & 7) (conflict-free 8-byte writes by token and 16-byte reads by row).
    __syncthreads();
    uint8_t* s_y = s_xT;
    {
      // this lane's rows are 32 jt + pc, so j & 7 = pc & 7 for both j-blocks
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
      // thread: token rows 32 k + t / 8 (k = 0..7), 16-byte column t % 8; (t / 8) & 7 is the
      // row's swizzle for every k
      const int jt8 = t >> 3, col = t & 7;
      const uint8_t* src = s_y + jt8 * 128 + ((col ^ (jt8 & 7)) * 16);
      const __amdgpu_buffer_rsrc_t yrs = buffer_rsrc(y + tok0 * HP + (size_t)h * kP);
      const uint32_t yo = (uint32_t)(jt8 * HP * 2 + col * 16);
      if (fs.stream) {
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

hipError_t launch_chunk_scan(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                             int dt_softplus, const float* A, const int8_t* cq_frag,
                             const float* C_scale, int c_per_token, const int8_t* pin,
                             const int8_t* cbq, const float* cb_scale, const float* state_scale,
                             const float* D, const float* corr, void* y, int y_dtype,
                             int32_t* y1_tap, int stream, hipStream_t st,
                             hipEvent_t ev_start, hipEvent_t ev_stop) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.nheads;
  if (nwork == 0) return hipSuccess;
  const dim3 grid((unsigned)nwork), block(256);
  FusedState fs;
  fs.stream = stream;
#define SSDI8_SCAN_ARGS(XT, YT)                                                                  \
  static_cast<const XT*>(x), dt, A, cq_frag, C_scale, c_per_token, const_cast<int8_t*>(pin),    \
      cbq, cb_scale, state_scale, D, corr, dt_softplus, static_cast<YT*>(y), y1_tap, d.seqlen,   \
      d.nheads, d.ngroups, d.nchunks, fs
#define SSDI8_SCAN_LAUNCH(XT, YT)                                                                \
  do {                                                                                           \
    if (ev_start || ev_stop)                                                                     \
      hipExtLaunchKernelGGL((chunk_scan_kernel<XT, YT, 0>), grid, block, 0, st, ev_start,        \
                            ev_stop, 0, SSDI8_SCAN_ARGS(XT, YT));                                \
    else                                                                                         \
      hipLaunchKernelGGL((chunk_scan_kernel<XT, YT, 0>), grid, block, 0, st,                     \
                         SSDI8_SCAN_ARGS(XT, YT));                                               \
  } while (0)
  if (x_dtype == 1 && y_dtype == 1) SSDI8_SCAN_LAUNCH(_Float16, _Float16);
  else if (x_dtype == 1) SSDI8_SCAN_LAUNCH(_Float16, float);
  else if (y_dtype == 1) SSDI8_SCAN_LAUNCH(float, _Float16);
  else SSDI8_SCAN_LAUNCH(float, float);
#undef SSDI8_SCAN_LAUNCH
#undef SSDI8_SCAN_ARGS
  return hipGetLastError();
}

hipError_t launch_chunk_scan_fused(const LayerDims& d, const _Float16* x, const float* dt,
                                   int dt_softplus, const float* A, const int8_t* cq_frag,
                                   const float* C_scale, int c_per_token, int8_t* pin,
                                   const int8_t* cbq, const float* cb_scale,
                                   const float* state_scale, const float* D, const float* corr,
                                   void* y, int y_dtype, const FusedState& fs, hipStream_t st,
                                   hipEvent_t ev_start, hipEvent_t ev_stop) {
  const int64_t nwork = (int64_t)d.batch * d.nchunks * d.nheads;
  if (nwork == 0) return hipSuccess;
  const dim3 grid((unsigned)nwork), block(256);
#define SSDI8_FUSED_ARGS(YT)                                                                     \
  x, dt, A, cq_frag, C_scale, c_per_token, pin, cbq, cb_scale, state_scale, D, corr, dt_softplus, \
      static_cast<YT*>(y), nullptr, d.seqlen, d.nheads, d.ngroups, d.nchunks, fs
#define SSDI8_FUSED_LAUNCH(YT, M)                                                                \
  do {                                                                                           \
    if (ev_start || ev_stop)                                                                     \
      hipExtLaunchKernelGGL((chunk_scan_kernel<_Float16, YT, M>), grid, block, 0, st, ev_start,  \
                            ev_stop, 0, SSDI8_FUSED_ARGS(YT));                                   \
    else                                                                                         \
      hipLaunchKernelGGL((chunk_scan_kernel<_Float16, YT, M>), grid, block, 0, st,               \
                         SSDI8_FUSED_ARGS(YT));                                                  \
  } while (0)
  if (y_dtype == 1 && fs.speculate) SSDI8_FUSED_LAUNCH(_Float16, 2);
  else if (y_dtype == 1) SSDI8_FUSED_LAUNCH(_Float16, 1);
  else if (fs.speculate) SSDI8_FUSED_LAUNCH(float, 2);
  else SSDI8_FUSED_LAUNCH(float, 1);
#undef SSDI8_FUSED_LAUNCH
#undef SSDI8_FUSED_ARGS
  return hipGetLastError();
}

}  // namespace ssdi8
