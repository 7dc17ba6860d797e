"""fp64 unquantized Mamba-2 SSD layer in three equivalent forms (oracle; test infrastructure).

Problem statement (Sec. 4.1): x (B,L,H,P), dt (B,L,H), A (H), B and C (B,L,G,N), output Y
(B,L,H,P).  B and C live on G groups and are broadcast to the H heads; head h reads group
h // (H/G) (contiguous heads per group, the Mamba-2 convention).  dt is the post-softplus
time step.  D is the per-head skip term of Mamba-2 (absent from Alg. 2, added to all forms).

  * recurrence  the discretised SSM run token by token (Eq. 2 with the zero-order-hold
                discretisation of A, Sec. 3.2):
                    h_t = exp(dt_t A) h_{t-1} + dt_t x_t B_t^T,   y_t = h_t C_t + D x_t
  * quadratic   the "attention" dual: Y = (M o C B^T) X + D X with the lower-triangular
                semiseparable mask M[t,s] = exp(cs_t - cs_s) dt_s for s <= t, cs = cumsum(dt A)
                (Sec. 4.1, first paragraph).
  * chunked     the five modules ChunkCumsum, ChunkState (Eq. 4), StatePassing (Eq. 5-6),
                ChunkBMM and ChunkScan 1/2 of Alg. 2.  Readings where the printed algorithm is
                loose: ChunkScan1 uses the state ENTERING the chunk (the result of passing up to
                the previous chunk) and its decay is exp(dA_cs) without a dt factor; ChunkScan2
                uses dt of the source (column) token and the causal mask i <= j.  With these
                readings the chunked form equals the recurrence, which the tests check.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np


def softplus64(v) -> np.ndarray:
    """softplus(v) = log(1 + exp(v)) in fp64, returning v itself above 20 (Alg. 2, module 1)."""
    v = np.asarray(v, np.float64)
    return np.where(v > 20.0, v, np.log1p(np.exp(np.minimum(v, 20.0))))


def head_group(nheads: int, ngroups: int) -> np.ndarray:
    """Group index read by each head: h // (H/G)."""
    assert nheads % ngroups == 0
    return np.arange(nheads) // (nheads // ngroups)


def ssd_recurrence(x, dt, A, B, C, D=None, init=None) -> Dict[str, np.ndarray]:
    """Token-by-token fp64 recurrence.  Pure loop over time; meant for tiny inputs."""
    x = np.asarray(x, np.float64)
    dt = np.asarray(dt, np.float64)
    A = np.asarray(A, np.float64)
    Bt, L, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    gi = head_group(H, G)
    Bh = np.asarray(B, np.float64)[:, :, gi, :]          # (Bt,L,H,N)
    Ch = np.asarray(C, np.float64)[:, :, gi, :]
    h = np.zeros((Bt, H, P, N)) if init is None else np.array(init, np.float64)
    y = np.empty((Bt, L, H, P))
    for t in range(L):
        a = np.exp(dt[:, t, :] * A[None, :])             # (Bt,H)
        h = a[:, :, None, None] * h + (dt[:, t, :, None, None] * x[:, t, :, :, None]
                                       * Bh[:, t, :, None, :])
        y[:, t] = np.einsum("bhpn,bhn->bhp", h, Ch[:, t])
    if D is not None:
        y = y + np.asarray(D, np.float64)[None, None, :, None] * x
    return {"y": y, "final_state": h}


def ssd_quadratic(x, dt, A, B, C, D=None, init=None) -> Dict[str, np.ndarray]:
    """Quadratic (attention) form with the full L x L semiseparable mask.  Tiny inputs only."""
    x = np.asarray(x, np.float64)
    dt = np.asarray(dt, np.float64)
    A = np.asarray(A, np.float64)
    Bt, L, H, P = x.shape
    G = B.shape[2]
    gi = head_group(H, G)
    B64 = np.asarray(B, np.float64)
    C64 = np.asarray(C, np.float64)
    y = np.empty((Bt, L, H, P))
    tt, ss = np.meshgrid(np.arange(L), np.arange(L), indexing="ij")
    causal = ss <= tt
    for b in range(Bt):
        for h in range(H):
            cs = np.cumsum(dt[b, :, h] * A[h])
            seg = np.where(causal, cs[:, None] - cs[None, :], -np.inf)
            M = np.exp(seg) * dt[b, None, :, h]
            CB = C64[b, :, gi[h]] @ B64[b, :, gi[h]].T       # (L,L): C_t . B_s
            y[b, :, h] = (M * CB) @ x[b, :, h]
            if init is not None:
                y[b, :, h] += np.exp(cs)[:, None] * (C64[b, :, gi[h]] @ np.asarray(
                    init, np.float64)[b, h].T)
    if D is not None:
        y = y + np.asarray(D, np.float64)[None, None, :, None] * x
    return {"y": y}


def ssd_chunked(x, dt, A, B, C, D=None, chunk: int = 256, init=None) -> Dict[str, np.ndarray]:
    """Alg. 2 in fp64 (no quantization).  Returns y plus the per-chunk intermediates:
    dA_cs (Bt,H,c,Q), chunk-local states (Bt,c,H,P,N), entering states (Bt,c,H,P,N),
    final state (Bt,H,P,N)."""
    x = np.asarray(x, np.float64)
    dt = np.asarray(dt, np.float64)
    A = np.asarray(A, np.float64)
    Bt, L, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    Q = chunk
    assert L % Q == 0
    nc = L // Q
    gi = head_group(H, G)
    # (Bt,c,Q,...) chunk views
    xc = x.reshape(Bt, nc, Q, H, P)
    dtc = dt.reshape(Bt, nc, Q, H)
    Bc = np.asarray(B, np.float64).reshape(Bt, nc, Q, G, N)[:, :, :, gi]   # (Bt,c,Q,H,N)
    Cc = np.asarray(C, np.float64).reshape(Bt, nc, Q, G, N)[:, :, :, gi]
    # Module 1 ChunkCumsum
    dA_cs = np.cumsum(dtc * A[None, None, None, :], axis=2)                # (Bt,c,Q,H)
    # Module 2 ChunkState: State = X^T (B o LUT_state), LUT_state = dt * exp(cs_last - cs)
    lut_state = dtc * np.exp(dA_cs[:, :, -1:, :] - dA_cs)
    states = np.einsum("bcqhp,bcqhn->bchpn", xc, Bc * lut_state[..., None])
    # Module 3 StatePassing: S_acc[c] = S[c] + exp(cs_last[c]) S_acc[c-1]
    decay_pass = np.exp(dA_cs[:, :, -1, :])                               # (Bt,c,H)
    entering = np.empty_like(states)
    run = np.zeros((Bt, H, P, N)) if init is None else np.array(init, np.float64)
    for c in range(nc):
        entering[:, c] = run
        run = states[:, c] + decay_pass[:, c, :, None, None] * run
    # Module 4 ChunkBMM: CB[c] = C_c B_c^T  (per head here, i.e. after the group broadcast)
    CB = np.einsum("bcjhn,bcihn->bchji", Cc, Bc)                         # (Bt,c,H,Q,Q)
    # Module 5 ChunkScan1: (C_j . S_in) * exp(cs_j)
    out_off = np.einsum("bcjhn,bchpn->bcjhp", Cc, entering) * np.exp(dA_cs)[..., None]
    # Module 6 ChunkScan2: (CB o LUT_scan2) X, LUT_scan2[j,i] = dt_i exp(cs_j - cs_i), i <= j
    jj, ii = np.meshgrid(np.arange(Q), np.arange(Q), indexing="ij")
    causal = ii <= jj
    csh = np.moveaxis(dA_cs, 3, 2)                                        # (Bt,c,H,Q)
    seg = np.where(causal, csh[..., :, None] - csh[..., None, :], -np.inf)
    lut2 = np.exp(seg) * np.moveaxis(dtc, 3, 2)[..., None, :]
    out_diag = np.einsum("bchji,bcihp->bcjhp", CB * lut2, xc)
    y = (out_off + out_diag).reshape(Bt, L, H, P)
    if D is not None:
        y = y + np.asarray(D, np.float64)[None, None, :, None] * x
    return {"y": y, "dA_cs": np.moveaxis(dA_cs, 3, 2), "states": states,
            "entering": entering, "final_state": run}


def chunk_states_fp64(x_bh, dt_bh, A_h, B_g, chunk: int):
    """fp64 chunk-local states of one (batch, head) sequence, (c,P,N), Eq. 4.  Used by
    calibration on full-size draws without materialising the (B,c,H,Q,Q) tensors."""
    L, P = x_bh.shape
    nc = L // chunk
    x = np.asarray(x_bh, np.float64).reshape(nc, chunk, P)
    dt = np.asarray(dt_bh, np.float64).reshape(nc, chunk)
    Bv = np.asarray(B_g, np.float64).reshape(nc, chunk, -1)
    cs = np.cumsum(dt * float(A_h), axis=1)
    lut = dt * np.exp(cs[:, -1:] - cs)
    states = np.matmul(np.swapaxes(x, 1, 2), Bv * lut[..., None])
    return states, np.exp(cs[:, -1]), cs


def ssd_chunked_bh(x_bh, dt_bh, A_h, B_g, C_g, D_h, chunk: int) -> Dict[str, np.ndarray]:
    """Alg. 2 in fp64 for one (batch, head) sequence: y (L,P), entering states (c,P,N), final.
    Same arithmetic as ssd_chunked, restricted to one slab to bound memory at full sizes."""
    L, P = x_bh.shape
    Q = chunk
    nc = L // Q
    states, decay_pass, cs = chunk_states_fp64(x_bh, dt_bh, A_h, B_g, Q)
    entering = np.empty_like(states)
    run = np.zeros(states.shape[1:])
    for c in range(nc):
        entering[c] = run
        run = states[c] + decay_pass[c] * run
    x = np.asarray(x_bh, np.float64).reshape(nc, Q, P)
    dt = np.asarray(dt_bh, np.float64).reshape(nc, Q)
    Bv = np.asarray(B_g, np.float64).reshape(nc, Q, -1)
    Cv = np.asarray(C_g, np.float64).reshape(nc, Q, -1)
    out_off = np.matmul(Cv, np.swapaxes(entering, 1, 2)) * np.exp(cs)[..., None]
    jj, ii = np.meshgrid(np.arange(Q), np.arange(Q), indexing="ij")
    seg = np.where(ii <= jj, cs[:, :, None] - cs[:, None, :], -np.inf)
    lut2 = np.exp(seg) * dt[:, None, :]
    CB = np.matmul(Cv, np.swapaxes(Bv, 1, 2))
    out_diag = np.matmul(CB * lut2, x)
    y = (out_off + out_diag).reshape(L, P) + float(D_h) * np.asarray(x_bh, np.float64)
    return {"y": y, "states": states, "entering": entering, "final_state": run, "CB": CB}
