/*
 * ssdi8.h — C ABI of the MI355X (gfx950) INT8 SSD chunk-scan library (libssdi8.so).
 *
 * The library computes the persistent-INT8 Mamba-2 SSD layer of "SSDi8: Accurate and Efficient
 * 8-bit Quantization for State Space Duality": B and C quantized once per group (Sec. 4.2,
 * "Quantization of B, C"), the chunk state as an INT8 x INT8 product after moving the decay
 * table onto x (Eq. 7) with an INT32->INT8 requantisation (Eq. 8), INT8 state passing with a
 * fixed-point decay and a k-bit shift (Eq. 9), INT8 ChunkBMM, INT8 ChunkScan1 with the decay
 * applied after the product, FP16 ChunkScan2 with the CB dequant scale folded into its table,
 * and an output epilogue adding the Mamba-2 D skip term and the per-channel correction term c of
 * Eq. 10.
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers owned by the caller; the library never allocates or
 *     frees device memory.  Scratch space is the caller's `workspace` (see
 *     ssdi8_ssd_workspace_size).
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = the default stream) and
 *     enqueues its kernels in order on that stream.  There is no hidden device synchronisation
 *     and no global mutable state: calls on different streams are independent.
 *   - All arguments are validated on the host BEFORE anything is enqueued; on any error nothing
 *     is launched and no output is touched.  Launch failures return SSDI8_ERR_HIP.  Device-side
 *     faults surface at the caller's next synchronisation.  Nothing is thrown across the ABI.
 *   - Layouts are dense row-major (C order) in the paper's storage order (Sec. 4.1):
 *     x, y [b, l, h, p];  dt [b, l, h];  A, D [h];  B, C [b, l, g, n].  Head h reads group
 *     h / (H/G) (contiguous heads per group).
 *   - Quantized integers are symmetric int8 in [-127, 127] (-128 is never produced).  A step
 *     size ("scale") alpha maps an integer q to alpha * q (Eq. 1: alpha = absmax / 127).
 *   - Supported shapes: headdim P = 64, dstate N = 128, chunk Q = 256; seqlen a multiple of the
 *     chunk; nheads a multiple of ngroups.  Others return SSDI8_ERR_UNSUPPORTED / _SHAPE.
 *   - Floating-point inputs containing NaN or Inf give unspecified (but in-bounds) results.
 */
#ifndef SSDI8_H
#define SSDI8_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SSDI8_OK = 0,
  SSDI8_ERR_NULL = 1,         /* a required pointer is NULL                                  */
  SSDI8_ERR_SHAPE = 2,        /* inconsistent or negative sizes, L % chunk != 0, H % G != 0  */
  SSDI8_ERR_UNSUPPORTED = 3,  /* valid but not implemented (P != 64, N != 128, chunk != 256) */
  SSDI8_ERR_ALIGN = 4,        /* a tensor pointer is not 16-byte aligned                     */
  SSDI8_ERR_WORKSPACE = 5,    /* workspace NULL or smaller than ssdi8_ssd_workspace_size     */
  SSDI8_ERR_HIP = 6,          /* a kernel launch failed                                      */
  SSDI8_ERR_ARG = 7           /* an enum / flag / shift argument is out of range             */
} ssdi8_status;

typedef enum { SSDI8_F32 = 0, SSDI8_F16 = 1 } ssdi8_dtype;

/* Quantization granules of a logical [b, l, k, m] tensor. */
typedef enum {
  SSDI8_GRAN_TENSOR = 0,   /* one step for the whole tensor              scale[1]        */
  SSDI8_GRAN_GROUP = 1,    /* one step per k (B, C: per group)           scale[k]        */
  SSDI8_GRAN_CHANNEL = 2,  /* one step per (k, m) (x: per head, channel) scale[k*m]      */
  SSDI8_GRAN_TOKEN = 3     /* one step per (b, l, k)                     scale[b*l*k]    */
} ssdi8_gran;

typedef struct {
  int64_t batch, seqlen, nheads, headdim, ngroups, dstate, chunk;
} ssdi8_dims;

/*
 * ssdi8_quantize_act — uniform symmetric 8-bit quantization of an activation (Eq. 1).
 * Used for B and C once per layer, per group (Sec. 4.2 "Quantization of B, C"), before their
 * reuse by ChunkState, ChunkBMM and ChunkScan1.
 *
 *   src      device, [b, l, k, m] of src_dtype (SSDI8_F16 or SSDI8_F32), 16-byte aligned.
 *   gran     granule of one step size (ssdi8_gran).
 *   scale    device fp32 step sizes, one per granule (sizes above).
 *            compute_scale = 0: read (static calibration, the paper's setting);
 *            compute_scale = 1: written with fl32(absmax / 127) of each granule (1 for an
 *            all-zero granule), then used.  Dynamic TENSOR/GROUP/CHANNEL modes support at most
 *            8192 granules (SSDI8_ERR_UNSUPPORTED beyond); TOKEN mode any number.
 *   dst      device int8 [b, l, k, m], 16-byte aligned, not overlapping src:
 *            dst = clamp(rne(fl32(src * fl32(1 / scale))), -127, 127).  With compute_scale = 1
 *            it also holds partial maxima while the steps are computed, before the codes.
 *   b*l == 0 is valid: src and dst may then be NULL; nothing is quantized (dynamic
 *   TENSOR/GROUP/CHANNEL steps are set to 1, TOKEN has no steps).
 * Errors: NULL scale, NULL src/dst with b*l > 0, negative b/l, k or m < 1, bad dtype/gran,
 * misalignment (src, dst 16 bytes; scale 4 bytes).
 */
ssdi8_status ssdi8_quantize_act(const void* src, int src_dtype, int64_t b, int64_t l, int64_t k,
                                int64_t m, int gran, float* scale, int compute_scale, int8_t* dst,
                                void* stream);

/*
 * ssdi8_state_pass — INT8 StatePassing across chunks (Eq. 9, Alg. 2 module 3):
 *     P_in[0] = init (zeros if init_q is NULL)
 *     P_in[c+1] = clamp(S_q[c] + ((q_d[c] * P_in[c] + r) >> shift), -127, 127)
 * with r = 2^(shift-1) when shift_round != 0 and r = 0 otherwise, int32 arithmetic with an
 * arithmetic right shift.  One step size per (h, p) is shared by all chunks, which is what makes
 * the integer recurrence valid (Sec. 4.2).
 *
 *   state_q     device int8 [batch, nchunks, nheads, headdim, dstate]: chunk-local states.
 *   decay_q     device int16 [batch, nheads, nchunks]: Q(Decay) = rne(exp(dA_cs_last) 2^shift),
 *               normally in [0, 2^shift]; other values are used as given.
 *   shift       k in [1, 14] (the paper uses 7).
 *   init_q      device int8 [batch, nheads, headdim, dstate] or NULL.
 *   state_in_q  device int8 [batch, nchunks, nheads, headdim, dstate]: P_in[c], the state
 *               ENTERING chunk c (read by ChunkScan1 of chunk c).
 *   final_q     device int8 [batch, nheads, headdim, dstate] = P_in[nchunks], or NULL.
 *   final_state device fp32 same shape = fl32(final_q * state_scale[h, p]), or NULL
 *               (state_scale must then be non-NULL, [nheads, headdim]).
 * nchunks == 0 copies init (or zeros) to the final outputs.  Pointers 16-byte aligned.
 */
ssdi8_status ssdi8_state_pass(const int8_t* state_q, const int16_t* decay_q, int shift,
                              int shift_round, const int8_t* init_q, int8_t* state_in_q,
                              int8_t* final_q, float* final_state, const float* state_scale,
                              int64_t batch, int64_t nchunks, int64_t nheads, int64_t headdim,
                              int64_t dstate, void* stream);

/*
 * Arguments of ssdi8_ssd_chunk_scan (Alg. 2 with the SSDi8 quantization of Sec. 4.2).
 * Sizes come from ssdi8_dims: B = batch, L = seqlen, H = nheads, P = headdim, G = ngroups,
 * N = dstate, Q = chunk, c = L / Q.  All pointers are device pointers, 16-byte aligned.
 */
typedef struct {
  const void* x;  int x_dtype;        /* [B,L,H,P] fp16 or fp32                                  */
  const float* dt; int dt_softplus;   /* [B,L,H]; if dt_softplus, softplus is applied first      */
                                      /*   (fp64, threshold 20, rounded once to fp32)            */
  const float* A;                     /* [H] decay parameter (<= 0)                              */
  const int8_t* Bq;                   /* [B,L,G,N] from ssdi8_quantize_act, per-group steps      */
  const int8_t* Cq;                   /* [B,L,G,N] per-group steps, or per-token steps; or both  */
                                      /*   NULL with B, C given unquantized (fields at the end)  */
  const float* B_scale;               /* [G]                                                     */
  const float* C_scale;               /* [G], or [B,L,G] when c_per_token != 0                   */
  int c_per_token;
  const float* D;                     /* [H] skip term, or NULL (= 0)                            */
  const float* corr;                  /* [H,P] per-channel correction c (Eq. 10), or NULL (= 0)  */
  const float* xs_scale;              /* step of X_scaled = LUT_state * x (Eq. 7): [H,P], or [H] */
  int xs_per_head;                    /*   when xs_per_head != 0                                 */
  const float* state_scale;           /* [H,P] step of the int8 states (Eq. 8, shared over c)    */
  const float* cb_scale;              /* [G] step of the int8 C.B^T                              */
  int decay_shift;                    /* k of Eq. 9, in [1, 14]; the paper uses 7                */
  int shift_round;                    /* 1: add 2^(k-1) before the shift; 0: floor shift         */
  const int8_t* init_state_q;         /* [B,H,P,N] int8 initial state at state_scale, or NULL    */
  void* y; int y_dtype;               /* [B,L,H,P] output, fp16 or fp32                          */
  int8_t* final_state_q;              /* [B,H,P,N] or NULL                                       */
  float* final_state;                 /* [B,H,P,N] fp32 = final_state_q * state_scale, or NULL   */
  /* Optional intermediate outputs (NULL = not produced), in the layouts listed: */
  int8_t* xs_q;                       /* [B,L,H,P]   Q(X_scaled)                                 */
  int32_t* state_i32;                 /* [B,c,H,P,N] State_INT32 (Eq. 7)                         */
  int8_t* state_q;                    /* [B,c,H,P,N] State_INT8 (Eq. 8), chunk-local             */
  int16_t* decay_q;                   /* [B,H,c]     Q(Decay) (Eq. 9)                            */
  int8_t* state_in_q;                 /* [B,c,H,P,N] state entering each chunk after passing     */
  int32_t* cb_i32;                    /* [B,c,G,Q,Q] C.B^T int32, entries i <= j only            */
  int8_t* cb_q;                       /* [B,c,G,Q,Q] C.B^T int8, entries i <= j only             */
  int32_t* scan1_i32;                 /* [B,L,H,P]   C_q . P_in^T int32 (ChunkScan1 product)     */
  void* workspace; size_t workspace_bytes;
  /* Optional per-module timing: NULL, or 5 hipEvent_t handles created by the caller (with
     timing enabled), marking the start of ChunkBMM, ChunkState, StatePassing and ChunkScan and
     the end of ChunkScan (the module breakdown of the paper's latency figures).  Events 0 and 1
     are set by ChunkBMM's own dispatch (its start and end), events 3 and 4 by the ChunkScan
     kernel's (hipExtLaunchKernelGGL: the timestamps a profiler's kernel trace reports), event 2
     is recorded on `stream` after ChunkState.  Leave NULL when the call is captured into a
     HIP graph. */
  void* const* stage_events;
  /* Kernel path.  With fp16 x and none of the taps xs_q, state_i32, state_q, decay_q, scan1_i32,
     dt_post requested, ChunkState, StatePassing and ChunkScan can run as one single-pass kernel
     in which each chunk obtains the int8 state entering it from the chunks before it in its
     sequence through the workspace (a flag per chunk; Eq. 9 applied in chunk order, so every
     integer result and y are bit-identical to the separate kernels).  The state_in_q tap is
     served by either path.  0: automatic (the single pass where it is the faster one, which
     takes enough concurrent sequences to hide the serial hand-offs: batch * nheads >= 72 with
     at least 4 chunks, or >= 48 with at least 32); 1: always the separate kernels; 2: the
     single pass whenever eligible.
     With the single pass, events 1-2 of stage_events mark the end of ChunkBMM and 3-4 the
     single pass's own start and end. */
  int path;
  /* Alternative to Bq / Cq (both NULL then): the unquantized B, C [B,L,G,N] of bc_dtype
     (SSDI8_F16 or SSDI8_F32), quantized inside ChunkBMM with the static steps B_scale, C_scale
     (per group, or C per token with c_per_token) exactly as ssdi8_quantize_act does, so the
     results are identical to quantizing first and passing Bq / Cq; the row-major int8 B, C
     are then never written. */
  const void* B; const void* C; int bc_dtype;
  /* Optional intermediate output like the taps above (NULL = not produced; requesting it selects
     the separate kernels): [B,L,H] fp32 dt as the kernels use it, i.e. after the softplus when
     dt_softplus != 0 (Alg. 2 module 1: fl32 of the fp64 softplus, threshold 20). */
  float* dt_post;
  /* Optional device int (4-byte aligned), or NULL.  A single-pass workgroup waits for the
     states of earlier chunks of its sequence with a bounded poll (2^16 polls, tens of ms); a
     wait that runs out is counted here and the kernel still finishes, but y and the final
     states of that layer are then unspecified.  The count is set to 0 by the call's first
     kernel and is 0 after the separate kernels, which never wait.  Read it after the stream
     has reached the end of the call; non-zero means the results must not be used (the GPU was
     preempted or shared for longer than the bound). */
  int* hand_off_timeouts;
} ssdi8_scan_args;

/* Workspace bytes needed by ssdi8_ssd_chunk_scan for these sizes (0 on invalid sizes). */
size_t ssdi8_ssd_workspace_size(const ssdi8_dims* d);

/*
 * ssdi8_ssd_chunk_scan — one SSD layer: ChunkCumsum, ChunkState, StatePassing, ChunkBMM,
 * ChunkScan1 + ChunkScan2 and the output epilogue
 *     y = y_off + y_diag + D[h] x + corr[h, p]
 * (Alg. 2 modules 1-6, Eq. 7-9, Eq. 10 correction applied at the SSD output).  B and C arrive
 * either quantized (Bq, Cq from ssdi8_quantize_act with per-group steps) or unquantized (B, C
 * of bc_dtype with Bq = Cq = NULL); in the second form ChunkBMM quantizes each row with the
 * static steps B_scale, C_scale as it loads it (Sec. 4.2: B and C quantized once, before any
 * reuse), bit-identically to calling ssdi8_quantize_act first, and the row-major int8 copies
 * are never written.  Intermediates go through `workspace`.
 */
ssdi8_status ssdi8_ssd_chunk_scan(const ssdi8_dims* d, const ssdi8_scan_args* a, void* stream);

/*
 * ssdi8_ssd_chunk_scan_noalloc — ssdi8_ssd_chunk_scan for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments and results, with `workspace` NULL and `workspace_bytes` 0; the scratch is
 * the library's own static device array of 128 MiB (134217728 bytes), one per GPU, created with
 * the library's device code and held until the process ends.  The call allocates nothing; its
 * first call on a device looks up that device's copy of the array.
 * Limit: ssdi8_ssd_workspace_size(d) must not exceed 128 MiB (e.g. 65536 tokens x 24 heads,
 * 16384 tokens x 80 heads); larger sizes return SSDI8_ERR_WORKSPACE before anything is launched.
 * A non-NULL workspace returns SSDI8_ERR_ARG.
 * Every call on one GPU uses the same scratch: calls that overlap on a GPU (on different streams,
 * or from different threads without ordering) race and give unspecified results; calls ordered
 * on one stream are safe (each call clears what must start at zero without hipMemsetAsync, so it
 * can be captured in a graph).
 */
ssdi8_status ssdi8_ssd_chunk_scan_noalloc(const ssdi8_dims* d, const ssdi8_scan_args* a,
                                          void* stream);

/* 1 if ssdi8_ssd_chunk_scan with these arguments runs the single-pass kernel (see `path`), 0 if
   the separate kernels (or on invalid sizes).  Host only; launches nothing. */
int ssdi8_uses_single_pass(const ssdi8_dims* d, const ssdi8_scan_args* a);

/*
 * ssdi8_decode_step — one token of every (batch, head) sequence in the recurrent mode of the same
 * persistent int8 state: the chunked method with a chunk of one token (Sec. 4.2; Eq. 7-9; Eq. 10
 * correction at the SSD output).  With cs = dt·A:
 *     q_d = rne(exp(cs)·2^k),  X_q = Q(fl32(dt·x) / a_X),  S_q = requant(X_q B_q^T, m_S)
 *     y   = (C_q · state) a_C a_S exp(cs) + fp16(CB_q a_CB dt)·fp16(x) + D x + corr
 *     state <- sat(S_q + ((q_d·state + r) >> k))
 * where y reads the state entering the token.  The same scales as ssdi8_ssd_chunk_scan; B and C of
 * the token are quantized first (ssdi8_quantize_act with l = 1).  Sizes as ssdi8_ssd_chunk_scan
 * (headdim 64, dstate 128).  All device pointers; asynchronous on `stream`; no workspace.
 */
typedef struct {
  const void* x; int x_dtype;         /* [B,H,P] the token's x, fp16 or fp32                     */
  const float* dt; int dt_softplus;   /* [B,H]                                                    */
  const float* A;                     /* [H]                                                      */
  const int8_t* Bq; const int8_t* Cq; /* [B,G,N] the token's quantized B, C                       */
  const float* B_scale;               /* [G]                                                      */
  const float* C_scale;               /* [G], or [B,G] when c_per_token != 0                      */
  int c_per_token;
  const float* D;                     /* [H] or NULL (= 0)                                        */
  const float* corr;                  /* [H,P] or NULL (= 0)                                      */
  const float* xs_scale; int xs_per_head;   /* [H,P], or [H] when xs_per_head != 0             */
  const float* state_scale;           /* [H,P]                                                    */
  const float* cb_scale;              /* [G]                                                      */
  int decay_shift; int shift_round;   /* k in [1, 14]; 1: add 2^(k-1) before the shift            */
  int8_t* state_q;                    /* [B,H,P,N] in: state entering the token; out: after it    */
  void* y; int y_dtype;               /* [B,H,P] output, fp16 or fp32                             */
  float* state;                       /* [B,H,P,N] fp32 = new state_q * state_scale, or NULL      */
} ssdi8_decode_args;
ssdi8_status ssdi8_decode_step(int64_t batch, int64_t nheads, int64_t headdim, int64_t ngroups,
                               int64_t dstate, const ssdi8_decode_args* a, void* stream);

/*
 * ssdi8_ssd_chunk_scan_fp16 — the same SSD layer without quantization, as the FP16 baseline the
 * paper's speedups are quoted against (Alg. 2 with fp16 contraction operands, fp32 accumulation
 * and fp32 chunk states):
 *     S = fp16(LUT_state·x)^T B,  P_in[c+1] = exp(cs_last) P_in[c] + S[c],
 *     y = (C · fp16(P_in)) exp(cs) + fp16(C B^T · dt · exp(segsum)) · x + D x
 * Sizes as ssdi8_ssd_chunk_scan; B and C are the unquantized fp16 (or fp32) tensors.  Scratch
 * goes through `workspace` (ssdi8_fp16_workspace_size).  stage_events: NULL or 5 hipEvent_t,
 * all recorded on `stream` between the kernels: before ChunkBMM, ChunkState, StatePassing and
 * ChunkScan and after ChunkScan.
 */
typedef struct {
  const void* x; int x_dtype;         /* [B,L,H,P] fp16 or fp32                                   */
  const float* dt; int dt_softplus;   /* [B,L,H]                                                  */
  const float* A;                     /* [H]                                                      */
  const void* B; const void* C;       /* [B,L,G,N]                                                */
  int bc_dtype;                       /* dtype of B and C: SSDI8_F16 or SSDI8_F32                 */
  const float* D;                     /* [H] or NULL (= 0)                                        */
  const float* init_state;            /* [B,H,P,N] fp32 initial state, or NULL (= 0)              */
  void* y; int y_dtype;               /* [B,L,H,P] output, fp16 or fp32                           */
  float* final_state;                 /* [B,H,P,N] fp32, or NULL                                  */
  void* workspace; size_t workspace_bytes;
  void* const* stage_events;          /* NULL or 5 hipEvent_t (see above)                         */
} ssdi8_fp16_args;
size_t ssdi8_fp16_workspace_size(const ssdi8_dims* d);
ssdi8_status ssdi8_ssd_chunk_scan_fp16(const ssdi8_dims* d, const ssdi8_fp16_args* a,
                                       void* stream);

/*
 * ssdi8_calibrate — the static step sizes of ssdi8_ssd_chunk_scan and the per-channel mean
 * correction, computed on the device from one calibration draw (Sec. 5 setup: symmetric static
 * steps fixed offline; Eq. 10 / Alg. 1 for a single layer, damped by eta):
 *     B_scale[g], C_scale[g]  fl32(absmax / 127) of B, C per group (Eq. 1)
 *     xs_scale               fl32(absmax / 127) of X_scaled = fl32(LUT_state x) (Eq. 7), per
 *                            (h, p) or per h; bit-identical to the values ChunkState quantizes
 *     state_scale[h, p]      absmax over (b, c, n) of the chunk-local states (Eq. 4) and of the
 *                            states after each chunk (passing in fp64), / 127
 *     cb_scale[g]            absmax of the causal entries of C B^T over (b, c), / 127
 *     corr[h, p]             eta * mean over (b, l) of (Y_fp - Y_q): Y_fp the FP16 layer
 *                            (ssdi8_ssd_chunk_scan_fp16), Y_q the INT8 layer with the steps above,
 *                            decay_shift / shift_round as given and no correction
 * An absmax of 0 gives a step of 1.  The unquantized states are accumulated from
 * X_scaled split into two fp16 parts (about 22 significant bits) times fp16 B with fp32 sums;
 * C B^T uses fp16 C and B (fp32 inputs are rounded to fp16 there).  Sizes as ssdi8_ssd_chunk_scan;
 * no initial state.  All device pointers, 16-byte aligned (the step outputs 4-byte); outputs are
 * written, never read; asynchronous on `stream`; scratch through `workspace`
 * (ssdi8_calibrate_workspace_size, about 8·B·L·H·P bytes more than the two layers' workspaces).
 * Errors as ssdi8_ssd_chunk_scan; eta must be finite; B·L == 0 is SSDI8_ERR_SHAPE.
 */
typedef struct {
  const void* x; int x_dtype;         /* [B,L,H,P] fp16 or fp32                                   */
  const float* dt; int dt_softplus;   /* [B,L,H]                                                  */
  const float* A;                     /* [H]                                                      */
  const void* B; const void* C;       /* [B,L,G,N] unquantized                                    */
  int bc_dtype;                       /* SSDI8_F16 or SSDI8_F32                                   */
  const float* D;                     /* [H] or NULL (= 0)                                        */
  int xs_per_head;                    /* 1: xs_scale is [H]; 0: [H,P]                             */
  float eta;                          /* damping of the correction; the paper uses 0.15           */
  int decay_shift; int shift_round;   /* of the INT8 layer that gives Y_q                         */
  float* B_scale; float* C_scale;     /* [G] out                                                  */
  float* xs_scale;                    /* [H,P] or [H] out                                         */
  float* state_scale;                 /* [H,P] out                                                */
  float* cb_scale;                    /* [G] out                                                  */
  float* corr;                        /* [H,P] out                                                */
  void* workspace; size_t workspace_bytes;
} ssdi8_calib_args;
size_t ssdi8_calibrate_workspace_size(const ssdi8_dims* d);
ssdi8_status ssdi8_calibrate(const ssdi8_dims* d, const ssdi8_calib_args* a, void* stream);

/*
 * ssdi8_mfma_probe — measurement helper: the on-box peak rate of the matrix cores, the
 * denominator of a "fraction of measured MFMA peak" beside the datasheet one.  Launches `blocks`
 * workgroups (1..65535) of 4 wavefronts; each wavefront runs 4 independent chains of `iters`
 * MFMAs on register operands (int8 v_mfma_i32_32x32x32_i8 for SSDI8_PROBE_I8, fp16
 * v_mfma_f32_32x32x16_f16 for SSDI8_PROBE_F16).  out: device, 256·blocks int32 (int8) or fp32
 * values (written, meaningless).  *ops (host, may be NULL) receives the multiply-add count × 2 of
 * the launch; time it with events on `stream`.
 */
typedef enum { SSDI8_PROBE_I8 = 0, SSDI8_PROBE_F16 = 1 } ssdi8_probe_kind;
ssdi8_status ssdi8_mfma_probe(int kind, int64_t iters, int64_t blocks, void* out, int64_t* ops,
                              void* stream);

/* Static description of a status code. */
const char* ssdi8_status_string(int status);

/* Library version, e.g. "0.1.0". */
const char* ssdi8_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SSDI8_H */
