// C ABI of libssdi8 (declared in include/ssdi8.h): argument validation, workspace planning and
// in-order kernel launches on the caller's stream.
#include "ssdi8.h"

#include <hip/hip_runtime.h>

#include <mutex>

#include "common.hpp"
#include "frag.hpp"
#include "launch.hpp"

// Scratch of ssdi8_ssd_chunk_scan_noalloc: the workspace of a call that brings none.  One copy
// per GPU, held until the process ends; calls on one GPU share it.
constexpr size_t kNoAllocScratchBytes = (size_t)128 << 20;
static __device__ __attribute__((aligned(256))) unsigned char scratch[kNoAllocScratchBytes];

namespace {

// The device address of `scratch` on the current device, looked up once per device (host code
// must never pass the array's own name to a kernel: on the host it is a stand-in, not a device
// address).
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::call_once(g_scratch_once[dev], [dev]() {
    void* p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = p;
  });
  if (g_scratch_err[dev] != hipSuccess) return g_scratch_err[dev];
  *out = g_scratch_ptr[dev];
  return *out ? hipSuccess : hipErrorInvalidSymbol;
}

// Compute units of the current device, looked up once per device (0 if unknown).
std::once_flag g_cus_once[kMaxDevices];
int g_cus[kMaxDevices];

int device_cus() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 0;
  std::call_once(g_cus_once[dev], [dev]() {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      n = 0;
    g_cus[dev] = n;
  });
  return g_cus[dev];
}

using ssdi8::LayerDims;

constexpr int64_t kMaxDim = (int64_t)1 << 31;

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
bool aligned16_or_null(const void* p) { return p == nullptr || aligned16(p); }

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

struct Plan {
  size_t bqT, cq, sq, pin, cbq, qd, sync, nsync, total;
};

// Workspace regions (256-byte aligned), the int8 ones in the MFMA fragment order of frag.hpp:
// B_q^T and C_q per chunk, chunk-local and entering int8 states, the causal blocks of the int8
// C.B^T; then the int16 Q(Decay).
Plan plan_workspace(const ssdi8_dims* d) {
  const size_t B = (size_t)d->batch, L = (size_t)d->seqlen, H = (size_t)d->nheads;
  const size_t P = (size_t)d->headdim, G = (size_t)d->ngroups, N = (size_t)d->dstate;
  const size_t Q = (size_t)d->chunk, nc = L / Q;
  Plan p;
  size_t off = 0;
  p.bqT = off; off = round_up(off + B * L * G * N, 256);
  p.cq = off;  off = round_up(off + B * L * G * N, 256);
  p.sq = off;  off = round_up(off + B * nc * H * P * N, 256);
  p.pin = off; off = round_up(off + B * nc * H * P * N, 256);
  p.cbq = off; off = round_up(off + B * nc * G * (size_t)ssdi8::frag::kCbChunkBytes, 256);
  (void)Q;
  p.qd = off;  off = round_up(off + B * H * nc * sizeof(int16_t), 256);
  // single-pass hand-off: ticket counters, timed-out waits, one flag per (b, h, c)
  p.nsync = ssdi8::kSyncFlags + B * H * nc;
  p.sync = off; off = round_up(off + p.nsync * sizeof(int), 256);
  p.total = off;
  return p;
}

struct Fp16Plan {
  size_t bT, c16, S, pin, cb, dec, total;
};

// FP16-baseline workspace: fp16 B^T and C fragments per chunk, fp32 chunk states and entering
// states (fragment order), fp32 causal CB blocks, fp32 per-chunk decays.
Fp16Plan plan_fp16(const ssdi8_dims* d) {
  const size_t B = (size_t)d->batch, L = (size_t)d->seqlen, H = (size_t)d->nheads;
  const size_t P = (size_t)d->headdim, G = (size_t)d->ngroups, N = (size_t)d->dstate;
  const size_t nc = L / (size_t)d->chunk;
  Fp16Plan p;
  size_t off = 0;
  p.bT = off;  off = round_up(off + 2 * B * L * G * N, 256);
  p.c16 = off; off = round_up(off + 2 * B * L * G * N, 256);
  p.S = off;   off = round_up(off + 4 * B * nc * H * P * N, 256);
  p.pin = off; off = round_up(off + 4 * B * nc * H * P * N, 256);
  p.cb = off;  off = round_up(off + 4 * B * nc * G * (size_t)ssdi8::frag::kCbBlocks * 1024, 256);
  p.dec = off; off = round_up(off + 4 * B * H * nc, 256);
  p.total = off;
  return p;
}

struct CalibPlan {
  Fp16Plan f16;
  Plan i8;
  size_t f16_base, i8_base, bq, cq, yfp, yq, dec64, amax, part, total;
};

// Calibration workspace: the FP16 layer's and the INT8 layer's workspaces, the quantized B and C,
// the two fp32 outputs Y_fp and Y_q, the fp64 chunk decays, and the absmax words (x: H*P,
// states: H*P, C.B^T: G).
CalibPlan plan_calib(const ssdi8_dims* d) {
  const size_t B = (size_t)d->batch, L = (size_t)d->seqlen, H = (size_t)d->nheads;
  const size_t P = (size_t)d->headdim, G = (size_t)d->ngroups, N = (size_t)d->dstate;
  const size_t nc = L / (size_t)d->chunk;
  CalibPlan p;
  p.f16 = plan_fp16(d);
  p.i8 = plan_workspace(d);
  size_t off = 0;
  p.f16_base = off; off = round_up(off + p.f16.total, 256);
  p.i8_base = off;  off = round_up(off + p.i8.total, 256);
  p.bq = off;       off = round_up(off + B * L * G * N, 256);
  p.cq = off;       off = round_up(off + B * L * G * N, 256);
  p.yfp = off;      off = round_up(off + 4 * B * L * H * P, 256);
  p.yq = off;       off = round_up(off + 4 * B * L * H * P, 256);
  p.dec64 = off;    off = round_up(off + 8 * B * H * nc, 256);
  p.amax = off;     off = round_up(off + 4 * (2 * H * P + G), 256);
  p.part = off;     off = round_up(off + ssdi8::calib_corr_scratch_bytes((int)H), 256);
  p.total = off;
  return p;
}

ssdi8_status check_dims(const ssdi8_dims* d) {
  if (!d) return SSDI8_ERR_NULL;
  if (d->batch < 0 || d->seqlen < 0 || d->nheads < 1 || d->headdim < 1 || d->ngroups < 1 ||
      d->dstate < 1 || d->chunk < 1)
    return SSDI8_ERR_SHAPE;
  if (d->batch >= kMaxDim || d->seqlen >= kMaxDim || d->nheads >= kMaxDim ||
      d->ngroups >= kMaxDim)
    return SSDI8_ERR_SHAPE;
  if (d->nheads % d->ngroups != 0 || d->seqlen % d->chunk != 0) return SSDI8_ERR_SHAPE;
  if (d->headdim != ssdi8::kP || d->dstate != ssdi8::kN || d->chunk != ssdi8::kQ)
    return SSDI8_ERR_UNSUPPORTED;
  // element counts of the largest tensors must stay addressable and grids launchable
  const double xel = (double)d->batch * d->seqlen * d->nheads * d->headdim;
  if (xel > 4.0e12) return SSDI8_ERR_SHAPE;
  const double nwork = (double)d->batch * (d->seqlen / d->chunk) * d->nheads;
  if (nwork >= 2147483647.0) return SSDI8_ERR_SHAPE;
  // the kernels address one chunk of one head's x / y rows with 32-bit byte offsets
  if ((double)d->nheads * d->headdim * d->chunk * 4.0 >= 4294967296.0)
    return SSDI8_ERR_UNSUPPORTED;
  return SSDI8_OK;
}

// Whether ssdi8_ssd_chunk_scan runs ChunkState, StatePassing and ChunkScan as the single pass.
bool single_pass(const ssdi8_dims* d, const ssdi8_scan_args* a) {
  // the entering states (state_in_q) are in the workspace either way; the other taps are
  // intermediates only the separate kernels hold
  const bool eligible = a->x_dtype == SSDI8_F16 && !a->xs_q && !a->dt_post && !a->state_i32 &&
                        !a->state_q && !a->decay_q && !a->scan1_i32;
  if (!eligible) return false;
  if (a->path != 0) return a->path == 2;
  // automatic: the single pass hides its chains of hand-offs behind enough concurrent sequences.
  // Measured crossover on MI355X (130M-shaped layers, B H sequences of nc chunks), taken where
  // the chains are longest (slowly decaying heads, no chunk with a zero Q(Decay)): it wins from
  // 72 sequences at 4 chunks and more, and from 48 sequences at 32 chunks
  const int64_t nc = d->chunk > 0 ? d->seqlen / d->chunk : 0;
  const int64_t bh = d->batch * d->nheads;
  return (bh >= 72 && nc >= 4) || (bh >= 48 && nc >= 32);
}

}  // namespace

extern "C" {

int ssdi8_uses_single_pass(const ssdi8_dims* d, const ssdi8_scan_args* a) {
  if (check_dims(d) != SSDI8_OK || !a || a->path < 0 || a->path > 2) return 0;
  return single_pass(d, a) ? 1 : 0;
}

const char* ssdi8_version(void) { return "0.1.0"; }

const char* ssdi8_status_string(int s) {
  switch (s) {
    case SSDI8_OK: return "ok";
    case SSDI8_ERR_NULL: return "required pointer is NULL";
    case SSDI8_ERR_SHAPE: return "invalid or inconsistent sizes";
    case SSDI8_ERR_UNSUPPORTED: return "sizes not supported (need headdim 64, dstate 128, chunk 256)";
    case SSDI8_ERR_ALIGN: return "tensor pointer not 16-byte aligned";
    case SSDI8_ERR_WORKSPACE: return "workspace missing or too small";
    case SSDI8_ERR_HIP: return "HIP kernel launch failed";
    case SSDI8_ERR_ARG: return "argument out of range";
    default: return "unknown status";
  }
}

ssdi8_status ssdi8_quantize_act(const void* src, int src_dtype, int64_t b, int64_t l, int64_t k,
                                int64_t m, int gran, float* scale, int compute_scale, int8_t* dst,
                                void* stream) {
  if (src_dtype != SSDI8_F32 && src_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (gran < SSDI8_GRAN_TENSOR || gran > SSDI8_GRAN_TOKEN) return SSDI8_ERR_ARG;
  if (b < 0 || l < 0 || k < 1 || m < 1) return SSDI8_ERR_SHAPE;
  if (b >= kMaxDim || l >= kMaxDim || k >= kMaxDim || m >= kMaxDim) return SSDI8_ERR_SHAPE;
  if ((double)b * l * k * m > 4.0e12) return SSDI8_ERR_SHAPE;
  const bool empty = (b == 0 || l == 0);
  if (!scale || (!empty && (!src || !dst))) return SSDI8_ERR_NULL;
  if (!aligned16_or_null(src) || !aligned16_or_null(dst) || ((uintptr_t)scale & 3u))
    return SSDI8_ERR_ALIGN;
  if (compute_scale && gran != SSDI8_GRAN_TOKEN) {
    const int64_t ngran = gran == SSDI8_GRAN_TENSOR ? 1 : (gran == SSDI8_GRAN_GROUP ? k : k * m);
    if (ngran > ssdi8::quantize_max_granules()) return SSDI8_ERR_UNSUPPORTED;
  }
  hipError_t e = ssdi8::launch_quantize(src, src_dtype, b, l, k, m, gran, scale, compute_scale,
                                        dst, (hipStream_t)stream);
  return e == hipSuccess ? SSDI8_OK : SSDI8_ERR_HIP;
}

ssdi8_status ssdi8_state_pass(const int8_t* state_q, const int16_t* decay_q, int shift,
                              int shift_round, const int8_t* init_q, int8_t* state_in_q,
                              int8_t* final_q, float* final_state, const float* state_scale,
                              int64_t batch, int64_t nchunks, int64_t nheads, int64_t headdim,
                              int64_t dstate, void* stream) {
  if (batch < 0 || nchunks < 0 || nheads < 1 || headdim < 1 || dstate < 1)
    return SSDI8_ERR_SHAPE;
  if (batch >= kMaxDim || nchunks >= kMaxDim || nheads >= kMaxDim || headdim >= kMaxDim ||
      dstate >= kMaxDim)
    return SSDI8_ERR_SHAPE;
  if ((double)batch * nchunks * nheads * headdim * dstate > 4.0e12) return SSDI8_ERR_SHAPE;
  if (shift < 1 || shift > 14) return SSDI8_ERR_ARG;
  if (nchunks > 0 && (!state_q || !decay_q || !state_in_q)) return SSDI8_ERR_NULL;
  if (final_state && !state_scale) return SSDI8_ERR_NULL;
  if (dstate % 4 != 0) return SSDI8_ERR_UNSUPPORTED;
  if (!aligned16_or_null(state_q) || !aligned16_or_null(state_in_q) ||
      !aligned16_or_null(init_q) || !aligned16_or_null(final_q) ||
      !aligned16_or_null(final_state) || ((uintptr_t)decay_q & 1u))
    return SSDI8_ERR_ALIGN;
  hipError_t e = ssdi8::launch_state_pass(batch, nchunks, nheads, headdim * dstate, headdim,
                                          state_q, decay_q, shift, shift_round, init_q,
                                          state_in_q, nullptr, final_q, final_state, state_scale,
                                          0, (hipStream_t)stream);
  return e == hipSuccess ? SSDI8_OK : SSDI8_ERR_HIP;
}

size_t ssdi8_ssd_workspace_size(const ssdi8_dims* d) {
  if (check_dims(d) != SSDI8_OK) return 0;
  return plan_workspace(d).total;
}

ssdi8_status ssdi8_ssd_chunk_scan(const ssdi8_dims* d, const ssdi8_scan_args* a, void* stream) {
  ssdi8_status s = check_dims(d);
  if (s != SSDI8_OK) return s;
  if (!a) return SSDI8_ERR_NULL;
  if (a->x_dtype != SSDI8_F32 && a->x_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (a->y_dtype != SSDI8_F32 && a->y_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (a->decay_shift < 1 || a->decay_shift > 14) return SSDI8_ERR_ARG;
  if (a->path < 0 || a->path > 2) return SSDI8_ERR_ARG;
  const bool work = d->batch > 0 && d->seqlen > 0;
  // B, C: quantized (Bq, Cq) or unquantized (B, C with bc_dtype), not both, not a mix
  const bool quantized = a->Bq || a->Cq;
  if (quantized && (a->B || a->C)) return SSDI8_ERR_ARG;
  if (!quantized && (a->B || a->C) && a->bc_dtype != SSDI8_F32 && a->bc_dtype != SSDI8_F16)
    return SSDI8_ERR_ARG;
  const void* Bsrc = quantized ? (const void*)a->Bq : a->B;
  const void* Csrc = quantized ? (const void*)a->Cq : a->C;
  if (work && (!a->x || !a->dt || !a->A || !Bsrc || !Csrc || !a->B_scale || !a->C_scale ||
               !a->xs_scale || !a->state_scale || !a->cb_scale || !a->y))
    return SSDI8_ERR_NULL;
  if (a->final_state && !a->state_scale) return SSDI8_ERR_NULL;
  if ((uintptr_t)a->hand_off_timeouts & 3u) return SSDI8_ERR_ALIGN;
  const void* al[] = {a->x, a->y, a->Bq, a->Cq, a->B, a->C, a->init_state_q, a->final_state_q,
                      a->final_state, a->xs_q, a->state_i32, a->state_q, a->decay_q,
                      a->state_in_q, a->cb_i32, a->cb_q, a->scan1_i32, a->dt_post,
                      a->workspace};
  for (const void* p : al)
    if (!aligned16_or_null(p)) return SSDI8_ERR_ALIGN;
  const Plan plan = plan_workspace(d);
  if (work && (!a->workspace || a->workspace_bytes < plan.total)) return SSDI8_ERR_WORKSPACE;
  if (a->stage_events)
    for (int i = 0; i < 5; ++i)
      if (!a->stage_events[i]) return SSDI8_ERR_NULL;

  hipStream_t st = (hipStream_t)stream;
  LayerDims ld;
  ld.batch = (int)d->batch;
  ld.seqlen = (int)d->seqlen;
  ld.nheads = (int)d->nheads;
  ld.ngroups = (int)d->ngroups;
  ld.nchunks = (int)(d->seqlen / d->chunk);
  const int64_t elems = d->headdim * d->dstate;

  if (!work) {
    // no tokens: the final state is the initial state
    if (d->batch > 0 && (a->final_state_q || a->final_state)) {
      hipError_t e = ssdi8::launch_state_pass(d->batch, 0, d->nheads, elems, d->headdim,
                                              nullptr, nullptr, a->decay_shift, a->shift_round,
                                              a->init_state_q, nullptr, nullptr,
                                              a->final_state_q, a->final_state, a->state_scale,
                                              0, st);
      if (e != hipSuccess) return SSDI8_ERR_HIP;
    }
    return SSDI8_OK;
  }

  char* ws = static_cast<char*>(a->workspace);
  int8_t* bqT = reinterpret_cast<int8_t*>(ws + plan.bqT);
  int8_t* cq = reinterpret_cast<int8_t*>(ws + plan.cq);
  int8_t* sq = reinterpret_cast<int8_t*>(ws + plan.sq);
  int8_t* pin = reinterpret_cast<int8_t*>(ws + plan.pin);
  int8_t* cbq = reinterpret_cast<int8_t*>(ws + plan.cbq);
  int16_t* qd = a->decay_q ? a->decay_q : reinterpret_cast<int16_t*>(ws + plan.qd);

  // stage events: 0 and 1 are ChunkBMM's own start and end, 3 and 4 the ChunkScan (or single
  // pass) kernel's; 2 is recorded on the stream after ChunkState (after ChunkBMM on the single
  // pass), so StatePassing's share runs from it to ChunkScan's start
  hipEvent_t ev[5] = {};
  if (a->stage_events)
    for (int i = 0; i < 5; ++i) ev[i] = static_cast<hipEvent_t>(a->stage_events[i]);
  auto mark = [&](int i) -> bool {
    return !a->stage_events || hipEventRecord(ev[i], st) == hipSuccess;
  };
  const bool fused = single_pass(d, a);
  int* sync = reinterpret_cast<int*>(ws + plan.sync);
  hipError_t e = ssdi8::launch_chunk_bmm(ld, Csrc, Bsrc, quantized ? -1 : a->bc_dtype,
                                         a->C_scale, a->c_per_token,
                                         a->B_scale, a->cb_scale, cbq, a->cb_q, a->cb_i32, bqT,
                                         cq, fused ? 1 : 0, sync, fused ? (int)plan.nsync : 0,
                                         a->hand_off_timeouts, st, ev[0], ev[1]);
  if (e != hipSuccess) return SSDI8_ERR_HIP;
  if (fused) {
    if (!mark(2)) return SSDI8_ERR_HIP;
    ssdi8::FusedState fs;
    fs.bqT = bqT;
    fs.sq = sq;
    fs.B_scale = a->B_scale;
    fs.xs_scale = a->xs_scale;
    fs.xs_per_head = a->xs_per_head;
    fs.shift = a->decay_shift;
    fs.radd = a->shift_round ? (1 << (a->decay_shift - 1)) : 0;
    fs.init = a->init_state_q;
    fs.final_q = a->final_state_q;
    fs.final_state = a->final_state;
    fs.sync = sync;
    fs.timeouts = a->hand_off_timeouts;
    fs.nbh = ld.batch * ld.nheads;
    fs.nclass = ssdi8::sync_classes(fs.nbh);
    fs.spin_limit = 1 << 16;   // polls of ~1 us: a wait gives up after ~65 ms
    // at most two rounds of workgroups (four per CU): the first loads of every item wait in
    // full, so they are requested with the ticket for the item dispatch order predicts
    const int64_t nitems = (int64_t)ld.batch * ld.nchunks * ld.nheads;
    fs.speculate = nitems <= (int64_t)8 * device_cus() ? 1 : 0;
    fs.stream = ssdi8::stream_xy(ld, 2, a->y_dtype == SSDI8_F16 ? 2 : 4);
    e = ssdi8::launch_chunk_scan_fused(ld, static_cast<const _Float16*>(a->x), a->dt,
                                       a->dt_softplus, a->A, cq, a->C_scale, a->c_per_token, pin,
                                       cbq, a->cb_scale, a->state_scale, a->D, a->corr, a->y,
                                       a->y_dtype, fs, st, ev[3], ev[4]);
    if (e != hipSuccess) return SSDI8_ERR_HIP;
    if (a->state_in_q) {
      e = ssdi8::launch_pin_tap(pin, a->state_in_q, (int64_t)ld.batch * ld.nchunks * ld.nheads,
                                st);
      if (e != hipSuccess) return SSDI8_ERR_HIP;
    }
    return SSDI8_OK;
  }
  e = ssdi8::launch_chunk_state(ld, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, bqT,
                                a->B_scale, a->xs_scale, a->xs_per_head, a->state_scale,
                                a->decay_shift, sq, qd, a->xs_q, a->state_q, a->state_i32,
                                a->dt_post, st);
  if (e != hipSuccess || !mark(2)) return SSDI8_ERR_HIP;
  e = ssdi8::launch_state_pass(d->batch, ld.nchunks, d->nheads, elems, d->headdim, sq, qd,
                               a->decay_shift, a->shift_round, a->init_state_q, pin,
                               a->state_in_q, a->final_state_q, a->final_state, a->state_scale,
                               (int)d->dstate, st);
  if (e != hipSuccess) return SSDI8_ERR_HIP;
  e = ssdi8::launch_chunk_scan(ld, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, cq,
                               a->C_scale, a->c_per_token, pin, cbq, a->cb_scale, a->state_scale,
                               a->D, a->corr, a->y, a->y_dtype, a->scan1_i32,
                               ssdi8::stream_xy(ld, a->x_dtype == SSDI8_F16 ? 2 : 4,
                                                a->y_dtype == SSDI8_F16 ? 2 : 4),
                               st, ev[3], ev[4]);
  if (e != hipSuccess) return SSDI8_ERR_HIP;
  return SSDI8_OK;
}

ssdi8_status ssdi8_ssd_chunk_scan_noalloc(const ssdi8_dims* d, const ssdi8_scan_args* a,
                                          void* stream) {
  ssdi8_status s = check_dims(d);
  if (s != SSDI8_OK) return s;
  if (!a) return SSDI8_ERR_NULL;
  if (a->workspace || a->workspace_bytes) return SSDI8_ERR_ARG;
  if (plan_workspace(d).total > kNoAllocScratchBytes) return SSDI8_ERR_WORKSPACE;
  ssdi8_scan_args b = *a;
  if (d->batch > 0 && d->seqlen > 0) {
    void* ws = nullptr;
    if (scratch_address(&ws) != hipSuccess) return SSDI8_ERR_HIP;
    b.workspace = ws;
    b.workspace_bytes = kNoAllocScratchBytes;
  }
  return ssdi8_ssd_chunk_scan(d, &b, stream);
}

size_t ssdi8_fp16_workspace_size(const ssdi8_dims* d) {
  if (check_dims(d) != SSDI8_OK) return 0;
  return plan_fp16(d).total;
}

ssdi8_status ssdi8_ssd_chunk_scan_fp16(const ssdi8_dims* d, const ssdi8_fp16_args* a,
                                       void* stream) {
  ssdi8_status s = check_dims(d);
  if (s != SSDI8_OK) return s;
  if (!a) return SSDI8_ERR_NULL;
  if (a->x_dtype != SSDI8_F32 && a->x_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (a->y_dtype != SSDI8_F32 && a->y_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (a->bc_dtype != SSDI8_F32 && a->bc_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  const bool work = d->batch > 0 && d->seqlen > 0;
  if (work && (!a->x || !a->dt || !a->A || !a->B || !a->C || !a->y)) return SSDI8_ERR_NULL;
  const void* al[] = {a->x, a->y, a->B, a->C, a->init_state, a->final_state, a->workspace};
  for (const void* p : al)
    if (!aligned16_or_null(p)) return SSDI8_ERR_ALIGN;
  const Fp16Plan plan = plan_fp16(d);
  if (work && (!a->workspace || a->workspace_bytes < plan.total)) return SSDI8_ERR_WORKSPACE;
  if (a->stage_events)
    for (int i = 0; i < 5; ++i)
      if (!a->stage_events[i]) return SSDI8_ERR_NULL;
  hipStream_t st = (hipStream_t)stream;
  LayerDims ld;
  ld.batch = (int)d->batch;
  ld.seqlen = (int)d->seqlen;
  ld.nheads = (int)d->nheads;
  ld.ngroups = (int)d->ngroups;
  ld.nchunks = (int)(d->seqlen / d->chunk);
  if (!work) {
    if (d->batch > 0 && a->final_state) {
      // no tokens: the final state is the initial state (a pass over zero chunks)
      ld.nchunks = 0;
      hipError_t e = ssdi8::launch_fp16_pass(ld, nullptr, nullptr, a->init_state, nullptr,
                                             a->final_state, st);
      if (e != hipSuccess) return SSDI8_ERR_HIP;
    }
    return SSDI8_OK;
  }
  char* ws = static_cast<char*>(a->workspace);
  _Float16* bT = reinterpret_cast<_Float16*>(ws + plan.bT);
  _Float16* c16 = reinterpret_cast<_Float16*>(ws + plan.c16);
  float* S = reinterpret_cast<float*>(ws + plan.S);
  float* pin = reinterpret_cast<float*>(ws + plan.pin);
  float* cb = reinterpret_cast<float*>(ws + plan.cb);
  float* dec = reinterpret_cast<float*>(ws + plan.dec);
  auto mark = [&](int i) -> bool {
    return !a->stage_events ||
           hipEventRecord(static_cast<hipEvent_t>(a->stage_events[i]), st) == hipSuccess;
  };
  if (!mark(0)) return SSDI8_ERR_HIP;
  hipError_t e = ssdi8::launch_fp16_bmm(ld, a->C, a->B, a->bc_dtype, cb, bT, c16, nullptr, st);
  if (e != hipSuccess || !mark(1)) return SSDI8_ERR_HIP;
  e = ssdi8::launch_fp16_state(ld, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, bT, S, dec,
                               st);
  if (e != hipSuccess || !mark(2)) return SSDI8_ERR_HIP;
  e = ssdi8::launch_fp16_pass(ld, S, dec, a->init_state, pin, a->final_state, st);
  if (e != hipSuccess || !mark(3)) return SSDI8_ERR_HIP;
  e = ssdi8::launch_fp16_scan(ld, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, c16, pin, cb,
                              a->D, a->y, a->y_dtype, st);
  if (e != hipSuccess || !mark(4)) return SSDI8_ERR_HIP;
  return SSDI8_OK;
}

size_t ssdi8_calibrate_workspace_size(const ssdi8_dims* d) {
  if (check_dims(d) != SSDI8_OK || d->batch == 0 || d->seqlen == 0) return 0;
  return plan_calib(d).total;
}

ssdi8_status ssdi8_calibrate(const ssdi8_dims* d, const ssdi8_calib_args* a, void* stream) {
  ssdi8_status s = check_dims(d);
  if (s != SSDI8_OK) return s;
  if (d->batch == 0 || d->seqlen == 0) return SSDI8_ERR_SHAPE;
  if (!a) return SSDI8_ERR_NULL;
  if (a->x_dtype != SSDI8_F32 && a->x_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (a->bc_dtype != SSDI8_F32 && a->bc_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (a->decay_shift < 1 || a->decay_shift > 14) return SSDI8_ERR_ARG;
  if (!(a->eta == a->eta) || a->eta > 3.0e38f || a->eta < -3.0e38f) return SSDI8_ERR_ARG;
  if (!a->x || !a->dt || !a->A || !a->B || !a->C || !a->B_scale || !a->C_scale ||
      !a->xs_scale || !a->state_scale || !a->cb_scale || !a->corr)
    return SSDI8_ERR_NULL;
  const void* al[] = {a->x, a->B, a->C, a->workspace};
  for (const void* p : al)
    if (!aligned16_or_null(p)) return SSDI8_ERR_ALIGN;
  const void* al4[] = {a->B_scale, a->C_scale, a->xs_scale, a->state_scale, a->cb_scale,
                       a->corr};
  for (const void* p : al4)
    if (((uintptr_t)p & 3u) != 0) return SSDI8_ERR_ALIGN;
  const CalibPlan plan = plan_calib(d);
  if (!a->workspace || a->workspace_bytes < plan.total) return SSDI8_ERR_WORKSPACE;
  if (ssdi8::quantize_max_granules() < d->ngroups) return SSDI8_ERR_UNSUPPORTED;

  hipStream_t st = (hipStream_t)stream;
  LayerDims ld;
  ld.batch = (int)d->batch;
  ld.seqlen = (int)d->seqlen;
  ld.nheads = (int)d->nheads;
  ld.ngroups = (int)d->ngroups;
  ld.nchunks = (int)(d->seqlen / d->chunk);
  const int H = (int)d->nheads, G = (int)d->ngroups, P = (int)d->headdim;
  char* ws = static_cast<char*>(a->workspace);
  char* f16 = ws + plan.f16_base;
  _Float16* bT = reinterpret_cast<_Float16*>(f16 + plan.f16.bT);
  _Float16* c16 = reinterpret_cast<_Float16*>(f16 + plan.f16.c16);
  float* S = reinterpret_cast<float*>(f16 + plan.f16.S);
  float* pin16 = reinterpret_cast<float*>(f16 + plan.f16.pin);
  float* cb = reinterpret_cast<float*>(f16 + plan.f16.cb);
  float* dec = reinterpret_cast<float*>(f16 + plan.f16.dec);
  char* i8 = ws + plan.i8_base;
  int8_t* Bq = reinterpret_cast<int8_t*>(ws + plan.bq);
  int8_t* Cq = reinterpret_cast<int8_t*>(ws + plan.cq);
  float* yfp = reinterpret_cast<float*>(ws + plan.yfp);
  float* yq = reinterpret_cast<float*>(ws + plan.yq);
  double* dec64 = reinterpret_cast<double*>(ws + plan.dec64);
  uint32_t* xs_amax = reinterpret_cast<uint32_t*>(ws + plan.amax);
  uint32_t* s_amax = xs_amax + H * P;
  uint32_t* cb_amax = s_amax + H * P;

  // steps of B and C (dynamic per-group absmax), then the quantities the other steps are taken of
  hipError_t e = ssdi8::launch_calib_zero(xs_amax, 2 * H * P + G, st);
  if (e == hipSuccess)
    e = ssdi8::launch_quantize(a->B, a->bc_dtype, d->batch, d->seqlen, d->ngroups, d->dstate,
                               SSDI8_GRAN_GROUP, a->B_scale, 1, Bq, st);
  if (e == hipSuccess)
    e = ssdi8::launch_quantize(a->C, a->bc_dtype, d->batch, d->seqlen, d->ngroups, d->dstate,
                               SSDI8_GRAN_GROUP, a->C_scale, 1, Cq, st);
  if (e == hipSuccess)
    e = ssdi8::launch_calib_xs(ld, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, xs_amax, st);
  if (e == hipSuccess)
    e = ssdi8::launch_fp16_bmm(ld, a->C, a->B, a->bc_dtype, cb, bT, c16, cb_amax, st);
  if (e == hipSuccess)
    e = ssdi8::launch_calib_states(ld, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, bT, S,
                                   dec64, s_amax, st);
  if (e == hipSuccess)
    e = ssdi8::launch_calib_steps(xs_amax, s_amax, cb_amax, a->xs_scale, a->state_scale,
                                  a->cb_scale, H, G, a->xs_per_head, st);
  // Y_fp: the FP16 layer (its ChunkBMM outputs are already in place)
  if (e == hipSuccess)
    e = ssdi8::launch_fp16_state(ld, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, bT, S, dec,
                                 st);
  if (e == hipSuccess) e = ssdi8::launch_fp16_pass(ld, S, dec, nullptr, pin16, nullptr, st);
  if (e == hipSuccess)
    e = ssdi8::launch_fp16_scan(ld, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, c16, pin16,
                                cb, a->D, yfp, SSDI8_F32, st);
  // Y_q: the INT8 layer with the new steps and no correction, as ssdi8_ssd_chunk_scan runs it
  if (e != hipSuccess) return SSDI8_ERR_HIP;
  {
    ssdi8_scan_args la = {};
    la.x = a->x;
    la.x_dtype = a->x_dtype;
    la.dt = a->dt;
    la.dt_softplus = a->dt_softplus;
    la.A = a->A;
    la.Bq = Bq;
    la.Cq = Cq;
    la.B_scale = a->B_scale;
    la.C_scale = a->C_scale;
    la.D = a->D;
    la.xs_scale = a->xs_scale;
    la.xs_per_head = a->xs_per_head;
    la.state_scale = a->state_scale;
    la.cb_scale = a->cb_scale;
    la.decay_shift = a->decay_shift;
    la.shift_round = a->shift_round;
    la.y = yq;
    la.y_dtype = SSDI8_F32;
    la.workspace = i8;
    la.workspace_bytes = plan.i8.total;
    const ssdi8_status ls = ssdi8_ssd_chunk_scan(d, &la, stream);
    if (ls != SSDI8_OK) return ls;
  }
  if (e == hipSuccess)
    e = ssdi8::launch_calib_corr(yfp, yq, reinterpret_cast<double*>(ws + plan.part), a->corr,
                                 d->batch * d->seqlen, H, a->eta, st);
  return e == hipSuccess ? SSDI8_OK : SSDI8_ERR_HIP;
}

ssdi8_status ssdi8_mfma_probe(int kind, int64_t iters, int64_t blocks, void* out,
                              int64_t* ops, void* stream) {
  if (kind != SSDI8_PROBE_I8 && kind != SSDI8_PROBE_F16) return SSDI8_ERR_ARG;
  if (iters < 1 || blocks < 1 || blocks > 65535 || iters > ((int64_t)1 << 40)) return SSDI8_ERR_ARG;
  if (!out) return SSDI8_ERR_NULL;
  if (((uintptr_t)out & 3u) != 0) return SSDI8_ERR_ALIGN;
  if (ops) *ops = ssdi8::mfma_probe_ops(kind, iters, blocks);
  if (ssdi8::launch_mfma_probe(kind, iters, blocks, out, (hipStream_t)stream) != hipSuccess)
    return SSDI8_ERR_HIP;
  return SSDI8_OK;
}

ssdi8_status ssdi8_decode_step(int64_t batch, int64_t nheads, int64_t headdim, int64_t ngroups,
                               int64_t dstate, const ssdi8_decode_args* a, void* stream) {
  if (batch < 0 || nheads < 1 || headdim < 1 || ngroups < 1 || dstate < 1) return SSDI8_ERR_SHAPE;
  if (batch >= kMaxDim || nheads >= kMaxDim || ngroups >= kMaxDim) return SSDI8_ERR_SHAPE;
  if (nheads % ngroups != 0) return SSDI8_ERR_SHAPE;
  if ((double)batch * nheads >= 2147483647.0) return SSDI8_ERR_SHAPE;
  if (headdim != ssdi8::kP || dstate != ssdi8::kN) return SSDI8_ERR_UNSUPPORTED;
  if (!a) return SSDI8_ERR_NULL;
  if (a->x_dtype != SSDI8_F32 && a->x_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (a->y_dtype != SSDI8_F32 && a->y_dtype != SSDI8_F16) return SSDI8_ERR_ARG;
  if (a->decay_shift < 1 || a->decay_shift > 14) return SSDI8_ERR_ARG;
  if (batch == 0) return SSDI8_OK;
  if (!a->x || !a->dt || !a->A || !a->Bq || !a->Cq || !a->B_scale || !a->C_scale ||
      !a->xs_scale || !a->state_scale || !a->cb_scale || !a->state_q || !a->y)
    return SSDI8_ERR_NULL;
  if (!aligned16(a->Bq) || !aligned16(a->Cq) || !aligned16(a->state_q) ||
      !aligned16_or_null(a->state))
    return SSDI8_ERR_ALIGN;
  hipError_t e = ssdi8::launch_decode(
      batch, nheads, ngroups, a->x, a->x_dtype, a->dt, a->dt_softplus, a->A, a->Bq, a->Cq,
      a->B_scale, a->C_scale, a->c_per_token, a->D, a->corr, a->xs_scale, a->xs_per_head,
      a->state_scale, a->cb_scale, a->decay_shift, a->shift_round, a->state_q, a->y, a->y_dtype,
      a->state, (hipStream_t)stream);
  return e == hipSuccess ? SSDI8_OK : SSDI8_ERR_HIP;
}

}  // extern "C"
