"""Static scale calibration and single-layer mean correction (oracle; test infrastructure).

Setup (Sec. 5): symmetric, static quantization with step sizes fixed offline from a calibration
draw; mean correction with damping eta = 0.15.  Granularity (Sec. 4.2): B and C per group;
X_scaled per (head, channel) or per head; State per (head, channel); CB per group (it lives on G).
Eq. 10 / Alg. 1 restricted to one layer: c_p = eta * (mean_{b,l} Y_fp - mean_{b,l} Y_q) per
output channel (h, p), where Y_q is the quantized layer without correction.

Calibration targets
  alpha_B[g], alpha_C[g]  absmax of the fp32 values of B / C in group g, / 127 (fp32 division).
  alpha_Xs               absmax of X_scaled = LUT_state o x (the fp32 values the quantizer sees).
  alpha_S[h,p]           absmax over (b, c, n) of the fp64 unquantized chunk-local AND passed
                         states, so that the int8 accumulation rarely saturates; / 127.
  alpha_CB[g]            absmax of the causal (i <= j) entries of the fp64 C B^T per chunk; / 127.
Any absmax of 0 gives a step of 1.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from . import exact, int8

F32 = np.float32
F64 = np.float64


def _step64(absmax64) -> np.ndarray:
    a = (np.asarray(absmax64, F64) / 127.0).astype(F32)
    return np.where(a == 0, F32(1.0), a).astype(F32)


def calibrate(x, dt_in, A, B, C, D, *, chunk: int, dt_softplus: bool = True,
              xs_per_head: bool = False, eta: float = 0.15, k: int = 7,
              shift_round: bool = True) -> Dict[str, np.ndarray]:
    Bt, L, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    Q = chunk
    gi = exact.head_group(H, G)
    dt32 = int8.dt_post(dt_in, dt_softplus)
    B32 = np.asarray(B).astype(F32)
    C32 = np.asarray(C).astype(F32)
    alpha_B = int8.absmax_step(int8.granule_absmax(B32, "group"))
    alpha_C = int8.absmax_step(int8.granule_absmax(C32, "group"))

    xs_max = np.zeros((H, P), F32)
    st_max = np.zeros((H, P), F64)
    cb_max = np.zeros(G, F64)
    causal = np.tril(np.ones((Q, Q), bool))
    for b in range(Bt):
        for g in range(G):
            Cv = C32[b, :, g].astype(F64).reshape(-1, Q, N)
            Bv = B32[b, :, g].astype(F64).reshape(-1, Q, N)
            cb = np.matmul(Cv, np.swapaxes(Bv, 1, 2))
            cb_max[g] = max(cb_max[g], float(np.abs(np.where(causal, cb, 0)).max()))
        for h in range(H):
            cum = int8.chunk_cumsum(dt32[b, :, h], A[h], Q, k)
            xs = cum["lut"][:, :, None] * np.asarray(x[b, :, h]).astype(F32).reshape(-1, Q, P)
            xs_max[h] = np.maximum(xs_max[h], np.abs(xs).max(axis=(0, 1)))
            states, decay_pass, _ = exact.chunk_states_fp64(
                x[b, :, h], dt32[b, :, h].astype(F64), float(F32(A[h])), B32[b, :, gi[h]], Q)
            run = np.zeros((P, N))
            m = np.abs(states).max(axis=(0, 2))
            for c in range(states.shape[0]):
                run = states[c] + decay_pass[c] * run
                m = np.maximum(m, np.abs(run).max(axis=1))
            st_max[h] = np.maximum(st_max[h], m)
    alpha_Xs = (int8.absmax_step(xs_max.max(axis=1)) if xs_per_head
                else int8.absmax_step(xs_max))
    scales = {"alpha_B": alpha_B, "alpha_C": alpha_C, "alpha_Xs": alpha_Xs,
              "alpha_S": _step64(st_max), "alpha_CB": _step64(cb_max)}
    scales["corr"] = mean_correction(x, dt_in, A, B, C, D, scales, chunk=Q,
                                     dt_softplus=dt_softplus, eta=eta, k=k,
                                     shift_round=shift_round)
    return scales


def mean_correction(x, dt_in, A, B, C, D, scales, *, chunk: int, dt_softplus: bool = True,
                    eta: float = 0.15, k: int = 7, shift_round: bool = True) -> np.ndarray:
    """Eq. 10 closed form per output channel (h, p), damped by eta: corr = eta * mean(Y_fp - Y_q),
    means over (b, l); Y_fp is the fp64 chunked SSD, Y_q the quantized layer with corr = 0."""
    Bt, L, H, P = x.shape
    G = B.shape[2]
    gi = exact.head_group(H, G)
    dt32 = int8.dt_post(dt_in, dt_softplus)
    zero = np.zeros((H, P), F32)
    diff_sum = np.zeros((H, P), F64)
    Bq, _ = int8.quantize_act(B, "group", scales["alpha_B"])
    Cq, _ = int8.quantize_act(C, "group", scales["alpha_C"])
    B32 = np.asarray(B).astype(F32)
    C32 = np.asarray(C).astype(F32)
    for b in range(Bt):
        for h in range(H):
            yq = int8.ssdi8_forward(x[b:b + 1, :, h:h + 1], dt_in[b:b + 1, :, h:h + 1],
                                    np.asarray(A, F32)[h:h + 1], B[b:b + 1, :, gi[h]:gi[h] + 1],
                                    C[b:b + 1, :, gi[h]:gi[h] + 1], np.asarray(D, F32)[h:h + 1],
                                    zero[h:h + 1],
                                    _slice_scales(scales, h, int(gi[h])), chunk=chunk,
                                    dt_softplus=dt_softplus, k=k, shift_round=shift_round,
                                    Bq=Bq[b:b + 1, :, gi[h]:gi[h] + 1],
                                    Cq=Cq[b:b + 1, :, gi[h]:gi[h] + 1], want=("y64",))["y64"]
            yf = exact.ssd_chunked_bh(x[b, :, h], dt32[b, :, h].astype(F64), float(F32(A[h])),
                                      B32[b, :, gi[h]], C32[b, :, gi[h]], float(F32(D[h])),
                                      chunk)["y"]
            diff_sum[h] += (yf - yq[0, :, 0]).sum(axis=0)
    return (eta * diff_sum / (Bt * L)).astype(F32)


def _slice_scales(scales, h: int, g: int) -> Dict[str, np.ndarray]:
    axs = np.asarray(scales["alpha_Xs"], F32)
    return {"alpha_B": np.asarray(scales["alpha_B"], F32)[g:g + 1],
            "alpha_C": np.asarray(scales["alpha_C"], F32)[g:g + 1],
            "alpha_Xs": axs[h:h + 1],
            "alpha_S": np.asarray(scales["alpha_S"], F32)[h:h + 1],
            "alpha_CB": np.asarray(scales["alpha_CB"], F32)[g:g + 1]}
