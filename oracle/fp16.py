"""The unquantized FP16 SSD layer (test infrastructure: the oracle of the on-box FP16 baseline).

This is Alg. 2 without the SSDi8 quantization: the same five modules, with every contraction
operand in fp16 (the storage type of x, B, C), contractions accumulated in fp32 and the chunk
states kept in fp32 -- the FP16 Mamba-2 SSD that the paper compares against (Sec. 5, the "FP16"
rows of the latency tables).  Rounding points, in the module order of Alg. 2:

  dt, dA, cs, LUT_state     as in the INT8 path (module 1, Eq. 4): fl32 softplus, fl32 dA, an exact
                            fp64 in-chunk prefix sum, LUT = fl32(dt fl32(exp(cs_last - cs)))
  ChunkState (module 2)     X~ = fp16(fl32(LUT x)) ;  S = fl32(sum_j X~[j,p] B[j,n])
  StatePassing (module 3)   d = fl32(exp(cs_last)) ;  P_in[c+1] = fl32(d P_in[c] + S[c]) (one
                            rounding, an fma), P_in[0] = the initial state (0 by default)
  ChunkBMM (module 4)       CB = fl32(sum_n C[j,n] B[i,n])
  ChunkScan1 (module 5)     Y1 = fl32(sum_n C[j,n] fp16(P_in[p,n])) ;  y_off = Y1 fl32(exp(cs_j))
  ChunkScan2 (module 6)     W = fp16(CB[j,i] dt_i exp(cs_j - cs_i)), i <= j ;  y_diag = W x
  output                    y = y_off + y_diag + D x

Sums are formed exactly (fp64 over fp16/fp32 operands) and rounded once, so the reference does
not depend on a summation order.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from . import exact
from . import int8

F16, F32, F64 = np.float16, np.float32, np.float64


def _fl32(v) -> np.ndarray:
    return np.asarray(v, F64).astype(F32)


def ssd_fp16_slab(x_seq, dt32_seq, A_h, B_seq, C_seq, D_h, chunk: int, init=None):
    """One (batch, head) sequence.  x_seq (L,P) as stored (fp16 or fp32), dt32_seq (L,) post
    softplus fp32, B_seq / C_seq (L,N) of the head's group.  Returns y64 (L,P), the chunk states
    S (c,P,N) fp32, the entering states P_in (c,P,N) fp32 and the final state (P,N) fp32."""
    L, P = x_seq.shape
    N = B_seq.shape[1]
    Q = chunk
    nc = L // Q
    cum = int8.chunk_cumsum(dt32_seq, A_h, Q)
    x16 = np.asarray(x_seq).astype(F16).reshape(nc, Q, P)
    x32 = np.asarray(x_seq).astype(F32).astype(F64).reshape(nc, Q, P)
    B16 = np.asarray(B_seq).astype(F16).astype(F64).reshape(nc, Q, N)
    C16 = np.asarray(C_seq).astype(F16).astype(F64).reshape(nc, Q, N)
    # ChunkState: X~ = fp16(fl32(LUT x))
    xt = (cum["lut"][:, :, None] * np.asarray(x_seq).astype(F32).reshape(nc, Q, P)).astype(F32)
    xt16 = xt.astype(F16).astype(F64)
    S = _fl32(np.matmul(np.swapaxes(xt16, 1, 2), B16))                    # (c,P,N) fp32
    # StatePassing
    d = np.exp(cum["cs"][:, -1]).astype(F32)
    pin = np.empty((nc, P, N), F32)
    run = np.zeros((P, N), F32) if init is None else np.asarray(init, F32)
    for c in range(nc):
        pin[c] = run
        run = _fl32(F64(d[c]) * run.astype(F64) + S[c].astype(F64))
    # ChunkBMM
    CB = _fl32(np.matmul(C16, np.swapaxes(B16, 1, 2)))                    # (c,Q,Q)
    # ChunkScan1
    Y1 = _fl32(np.matmul(C16, np.swapaxes(pin.astype(F16).astype(F64), 1, 2)))   # (c,Q,P)
    y_off = Y1.astype(F64) * np.exp(cum["cs"]).astype(F32).astype(F64)[:, :, None]
    # ChunkScan2
    cs = cum["cs"]
    jj, ii = np.meshgrid(np.arange(Q), np.arange(Q), indexing="ij")
    seg = np.where((ii <= jj)[None], cs[:, :, None] - cs[:, None, :], -np.inf)
    W = (CB.astype(F64) * cum["dt"].astype(F64)[:, None, :] * np.exp(seg)).astype(F16)
    y_diag = np.matmul(W.astype(F64), x16.astype(F64))
    y64 = y_off + y_diag + float(F32(D_h)) * x32
    return {"y64": y64.reshape(L, P), "S": S, "pin": pin, "final": run, "CB": CB,
            "Y1": Y1.reshape(L, P)}


def ssd_fp16_forward(x, dt_in, A, B, C, D, *, chunk: int, dt_softplus: bool = True,
                     init=None, heads=None) -> Dict[str, np.ndarray]:
    """Whole layer (or the (b, h) slabs in `heads`).  x (B,L,H,P); dt_in (B,L,H); A, D (H);
    B, C (B,L,G,N); init (B,H,P,N) fp32 or None.  Returns y64 (B,L,H,P) and the final state
    (B,H,P,N), or per-slab dicts under "slabs" when `heads` is given."""
    Bt, L, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    gi = exact.head_group(H, G)
    dt32 = int8.dt_post(dt_in, dt_softplus)
    pairs = [(b, h) for b in range(Bt) for h in range(H)] if heads is None else list(heads)
    out: Dict[str, np.ndarray] = {}
    if heads is None:
        out["y64"] = np.zeros((Bt, L, H, P), F64)
        out["final_state"] = np.zeros((Bt, H, P, N), F32)
    slabs = {}
    for (b, h) in pairs:
        g = int(gi[h])
        r = ssd_fp16_slab(x[b, :, h], dt32[b, :, h], A[h], B[b, :, g], C[b, :, g], D[h], chunk,
                          None if init is None else init[b, h])
        if heads is None:
            out["y64"][b, :, h] = r["y64"]
            out["final_state"][b, h] = r["final"]
        else:
            slabs[(b, h)] = r
    if heads is not None:
        out["slabs"] = slabs
    return out
