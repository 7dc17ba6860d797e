// Host-side launchers of the libssdi8 kernels (internal; the public ABI is include/ssdi8.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ssdi8 {

// ev_start / ev_stop of the launchers that take them: NULL, or events set to the kernel's own
// start and end (hipExtLaunchKernelGGL: the dispatch's timestamps, the figures a profiler's
// kernel trace reports) rather than markers recorded between kernels.

// Sizes shared by the SSD-layer kernels (P = 64, N = 128, Q = 256 fixed).
struct LayerDims {
  int batch, seqlen, nheads, ngroups, nchunks;
};

int quantize_max_granules();

hipError_t launch_quantize(const void* src, int src_dtype, int64_t b, int64_t l, int64_t k,
                           int64_t m, int gran, float* scale, int compute_scale, int8_t* dst,
                           hipStream_t st);

// ChunkBMM (int8 C.B^T per chunk and group, causal, requantized) plus the operand copies the
// later kernels read, all in the fragment order of frag.hpp: CB_q (36 KB per chunk and group),
// B_q^T of the chunk ([n][j] as kslice order, ChunkState) and C_q of the chunk ([j][n] as
// kslice order, ChunkScan1; permuted kslice order with cq_perm, for the single pass).  The taps
// are row-major [j][i].  sync[0, nsync) is cleared (the ticket and flags of
// launch_chunk_scan_fused; nsync = 0 when that kernel does not follow).
// src_dtype < 0: C, B are the quantized int8 tensors; 1 / 0: unquantized fp16 / fp32, quantized
// here with the static steps C_scale, B_scale exactly as launch_quantize does.
hipError_t launch_chunk_bmm(const LayerDims& d, const void* C, const void* B, int src_dtype,
                            const float* C_scale, int c_per_token, const float* B_scale,
                            const float* cb_scale, int8_t* cbq_frag, int8_t* cbq_tap,
                            int32_t* cb32_tap, int8_t* bqT_frag, int8_t* cq_frag, int cq_perm,
                            int* sync, int nsync, int* timeouts, hipStream_t st,
                            hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

// ChunkCumsum + reformulated ChunkState (Eq. 7-8) and Q(Decay) (Eq. 9).
hipError_t launch_chunk_state(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                              int dt_softplus, const float* A, const int8_t* bqT,
                              const float* B_scale, const float* xs_scale, int xs_per_head,
                              const float* state_scale, int shift, int8_t* sq, int16_t* qd,
                              int8_t* xq_tap, int8_t* sq_tap, int32_t* s32_tap, float* dt_tap,
                              hipStream_t st);

// The entering states P_in[c] the single pass leaves in the workspace (permuted kslice order,
// one P x N slab per (b, c, h)) as the row-major [b, c, h, p, n] tap.
hipError_t launch_pin_tap(const int8_t* pin, int8_t* tap, int64_t nslabs, hipStream_t st);

// INT8 StatePassing (Eq. 9) over [b, c, h, elems] slabs with elems = P*N (any P*N % 4 == 0).
// frag_k = 0: S_q and P_in row-major; frag_k = N: both in kslice order with K = N (P, N
// multiples of 32).  init, final_q, final_state and pin_tap are row-major either way.
hipError_t launch_state_pass(int64_t batch, int64_t nchunks, int64_t nheads, int64_t elems,
                             int64_t headdim, const int8_t* sq, const int16_t* qd, int shift,
                             int shift_round, const int8_t* init, int8_t* pin, int8_t* pin_tap,
                             int8_t* final_q, float* final_state, const float* state_scale,
                             int frag_k, hipStream_t st);

// ChunkScan1 (int8) + ChunkScan2 (fp16) + output epilogue; C_q, P_in and CB_q in fragment order.
// stream: x and y read / written non-temporally (stream_xy).
hipError_t launch_chunk_scan(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                             int dt_softplus, const float* A, const int8_t* cq_frag,
                             const float* C_scale, int c_per_token, const int8_t* pin,
                             const int8_t* cbq, const float* cb_scale, const float* state_scale,
                             const float* D, const float* corr, void* y, int y_dtype,
                             int32_t* y1_tap, int stream, hipStream_t st,
                             hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

// Single pass of ChunkState, StatePassing and ChunkScan (fp16 x): one workgroup per (b, c, h)
// in ticket order; each computes its chunk's S_q, obtains P_in[c] from the chunks before it (the
// previous chunk's P_in[c] in pin slot c, or an earlier published entering state and the
// published S_q of the chunks in between, sq slots; permuted kslice order, as C_q), publishes
// P_in[c+1] (slot c + 1, or the final states) and runs ChunkScan1/2 with x still in LDS.  sync
// (int words, cleared beforehand by ChunkBMM): the ticket counter of sequence class x at
// x * kSyncLine (one 128-byte line each, so that the classes' atomics do not serialize on one
// line), the count of waits that ran out at kSyncWait, and from kSyncFlags + (b H + h) nc + c
// the flag word of chunk c (its Q(Decay) and whether its S_q and P_in[c+1] are published).
constexpr int kSyncLine = 32;
constexpr int kSyncMaxClasses = 64;
constexpr int kSyncWait = kSyncMaxClasses * kSyncLine;
constexpr int kSyncFlags = kSyncWait + kSyncLine;
// Sequence classes of a launch: the largest of 64, 32, 16, 8 that divides the B H sequences
// (every class then holds as many items as workgroups draw from it first), else 8.
inline int sync_classes(int nbh) {
  for (int k = kSyncMaxClasses; k > 8; k >>= 1)
    if (nbh % k == 0) return k;
  return 8;
}
struct FusedState {
  const int8_t* bqT = nullptr;
  int8_t* sq = nullptr;      // published chunk-local states, one P x N slab per (b, c, h)
  const float* B_scale = nullptr;
  const float* xs_scale = nullptr;
  int xs_per_head = 0;
  int shift = 7;
  int radd = 0;
  const int8_t* init = nullptr;
  int8_t* final_q = nullptr;
  float* final_state = nullptr;
  int* sync = nullptr;
  int* timeouts = nullptr;   // the caller's count of waits that ran out, or NULL
  int nbh = 0;
  int nclass = 8;       // sync_classes(nbh)
  int spin_limit = 0;
  int speculate = 0;    // request the predicted item's first loads with its ticket (small grids)
  int stream = 0;       // x and y non-temporal (stream_xy)
};
// Whether a layer's x and y (touched once by the scan kernels) are streamed through the caches
// instead of cached: when together they exceed the 256 MB Infinity Cache, caching them only
// displaces the tiles every head of a chunk re-reads; below it, they stay resident for whatever
// reads them next.
inline int stream_xy(const LayerDims& d, int x_bytes, int y_bytes) {
  const int64_t elems = (int64_t)d.batch * d.seqlen * d.nheads * 64;   // P = 64
  return elems * (x_bytes + y_bytes) > ((int64_t)256 << 20) ? 1 : 0;
}
hipError_t launch_chunk_scan_fused(const LayerDims& d, const _Float16* x, const float* dt,
                                   int dt_softplus, const float* A, const int8_t* cq_frag,
                                   const float* C_scale, int c_per_token, int8_t* pin,
                                   const int8_t* cbq, const float* cb_scale,
                                   const float* state_scale, const float* D, const float* corr,
                                   void* y, int y_dtype, const FusedState& fs, hipStream_t st,
                                   hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

// One-token decode step on the persistent int8 state (a chunk of one token), in place.
hipError_t launch_decode(int64_t batch, int64_t nheads, int64_t ngroups, const void* x,
                         int x_dtype, const float* dt, int dt_softplus, const float* A,
                         const int8_t* Bq, const int8_t* Cq, const float* B_scale,
                         const float* C_scale, int c_per_token, const float* D,
                         const float* corr, const float* xs_scale, int xs_per_head,
                         const float* state_scale, const float* cb_scale, int shift,
                         int shift_round, int8_t* state, void* y, int y_dtype, float* state_f32,
                         hipStream_t st);

// FP16 baseline: ChunkBMM (fp32 CB blocks, fp16 B^T and C fragments), ChunkState (fp32 states,
// per-chunk decay), fp32 state passing, ChunkScan.
hipError_t launch_fp16_bmm(const LayerDims& d, const void* C, const void* B, int dtype,
                           float* cb_frag, _Float16* bT_frag, _Float16* c_frag,
                           uint32_t* cb_amax, hipStream_t st);
hipError_t launch_fp16_state(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                             int dt_softplus, const float* A, const _Float16* bT_frag, float* S,
                             float* dec, hipStream_t st);
hipError_t launch_fp16_pass(const LayerDims& d, const float* S, const float* dec,
                            const float* init, float* pin, float* final_state, hipStream_t st);
hipError_t launch_fp16_scan(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                            int dt_softplus, const float* A, const _Float16* c_frag,
                            const float* pin, const float* cb, const float* D, void* y,
                            int y_dtype, hipStream_t st);

// Calibration (static steps and the mean correction): absmax words cleared by a fill kernel,
// absmax of X_scaled, fp states from split fp16 operands with their absmax, the steps, the
// correction from two fp32 layer outputs.
hipError_t launch_calib_zero(uint32_t* p, int n, hipStream_t st);
hipError_t launch_calib_xs(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                           int dt_softplus, const float* A, uint32_t* xs_amax, hipStream_t st);
hipError_t launch_calib_states(const LayerDims& d, const void* x, int x_dtype, const float* dt,
                               int dt_softplus, const float* A, const _Float16* bT_frag,
                               float* S, double* dec64, uint32_t* s_amax, hipStream_t st);
hipError_t launch_calib_steps(const uint32_t* xs_amax, const uint32_t* s_amax,
                              const uint32_t* cb_amax, float* aXs, float* aS, float* aCB, int H,
                              int G, int xs_per_head, hipStream_t st);
size_t calib_corr_scratch_bytes(int H);
hipError_t launch_calib_corr(const float* y_fp, const float* y_q, double* part, float* corr,
                             int64_t T, int H, float eta, hipStream_t st);

// MFMA peak probe (int8 32x32x32 for dtype 0, fp16 32x32x16 otherwise): `blocks` workgroups of
// 4 waves, each running 4 independent chains of `iters` MFMAs; one value per thread to `out`.
int64_t mfma_probe_ops(int dtype, int64_t iters, int64_t blocks);
hipError_t launch_mfma_probe(int dtype, int64_t iters, int64_t blocks, void* out, hipStream_t st);

}  // namespace ssdi8
