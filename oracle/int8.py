"""The quantized SSDi8 SSD path, stage by stage (oracle; test infrastructure).

Written from the paper: Eq. 1 (uniform symmetric quantizer), Sec. 4.2 (B/C quantized once per
group; sparse-aware reformulation Eq. 7; INT32->INT8 state requantisation Eq. 8; INT8 state
passing with a fixed-point decay and a k-bit shift Eq. 9; INT8 ChunkBMM with its dequant scale
folded into the ChunkScan2 table; INT8 ChunkScan1 with the decay applied after the product;
ChunkScan2 kept in FP16), and the per-channel correction term of Eq. 10.

Arithmetic conventions (the readings where the paper leaves the choice open):
  fl32(v)       one IEEE round-to-nearest-even to fp32;  fp32 products are single IEEE products.
  quant(v, a)   clamp(rne(fl32(v * fl32(1/a))), -127, 127): Eq. 1 with step a = absmax/127.
  step(absmax)  fl32(absmax / 127) in fp32, and 1 where absmax == 0.
  cumsum        the in-chunk prefix sum of fl32(dt*A), exact and then rounded once to fp64
                (plain fp64 accumulation is exact when the chunk's nonzero terms span few enough
                binades; otherwise the exact sum is formed with math.fsum).
  Decay_state   fl32(exp(cs_last - cs_j)) from fp64 exp;  LUT_state = fl32(dt * Decay_state).
  Q(Decay)      rne(exp(cs_last) * 2^k) as an integer in [0, 2^k]  (Eq. 9, S = 2^k).
  multipliers   m_S = fl32(a_X * a_B / a_S) and m_CB = fl32(a_C * a_B / a_CB), each product and
                quotient formed in fp64 (Eq. 8 with step sizes; a_S is the state's step size).
  shift         (q_d * s + 2^(k-1)) >> k  (round half up; `shift_round=False` gives the plain
                floor shift), then saturating add in int32.
  ChunkScan1    y_off[j,p] = Y1[j,p] * a_C * a_S[p] * exp(cs_j), fp64.
  ChunkScan2    W[j,i] = fp16(CB_q[j,i] * a_CB * dt_i * exp(cs_j - cs_i)) for i <= j (one rounding
                from fp64), y_diag = W . fp16(x) accumulated in fp64.
  output        y = y_off + y_diag + D x + corr, rounded once to the output dtype.

Head h reads group h // (H/G).  Layouts of the returned intermediates match the library's debug
outputs: X_q (B,L,H,P), S32 / S_q / P_in (B,c,H,P,N), q_d (B,H,c), CB32 / CB_q (B,c,G,Q,Q) with
zeros above the diagonal, Y1 (B,L,H,P).
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, Optional, Tuple

import numpy as np

from .exact import head_group, softplus64

QMAX = 127
F32 = np.float32
F64 = np.float64


# ----------------------------------------------------------------------------- Eq. 1 quantizer
def fl32(v) -> np.ndarray:
    return np.asarray(v, F64).astype(F32)


def step_inverse(alpha) -> np.ndarray:
    """fl32(1/alpha), one IEEE fp32 division."""
    return (F32(1.0) / np.asarray(alpha, F32)).astype(F32)


def quantize(v32, inv32) -> np.ndarray:
    """clamp(rne(fl32(v * inv)), -127, 127) -> int8.  v and inv are fp32."""
    p = np.asarray(v32, F32) * np.asarray(inv32, F32)
    assert p.dtype == F32
    return np.clip(np.rint(p), -QMAX, QMAX).astype(np.int8)


def absmax_step(absmax) -> np.ndarray:
    """Step size alpha = absmax/(2^(b-1)-1) with b = 8 (Eq. 1), in fp32; 1 for an all-zero granule."""
    a = np.asarray(absmax, F32) / F32(QMAX)
    return np.where(a == 0, F32(1.0), a).astype(F32)


GRANS = ("tensor", "group", "channel", "token")


def granule_absmax(src32: np.ndarray, gran: str) -> np.ndarray:
    """Absolute maximum per granule of a logical (b, l, k, m) tensor.
    tensor: one value; group: per k; channel: per (k, m); token: per (b, l, k)."""
    a = np.abs(np.asarray(src32, F32))
    if a.size == 0:
        shape = {"tensor": (), "group": (a.shape[2],), "channel": a.shape[2:],
                 "token": a.shape[:3]}[gran]
        return np.zeros(shape, F32)
    if gran == "tensor":
        return a.max()
    if gran == "group":
        return a.max(axis=(0, 1, 3))
    if gran == "channel":
        return a.max(axis=(0, 1))
    if gran == "token":
        return a.max(axis=3)
    raise ValueError(gran)


def _expand(alpha, gran: str) -> np.ndarray:
    a = np.asarray(alpha, F32)
    return {"tensor": lambda: a.reshape(1, 1, 1, 1), "group": lambda: a[None, None, :, None],
            "channel": lambda: a[None, None], "token": lambda: a[..., None]}[gran]()


def quantize_act(src, gran: str, alpha=None) -> Tuple[np.ndarray, np.ndarray]:
    """Quantize a (b, l, k, m) activation; dynamic step sizes (absmax/127) when alpha is None."""
    src32 = np.asarray(src).astype(F32)
    if alpha is None:
        alpha = absmax_step(granule_absmax(src32, gran))
    q = quantize(src32, _expand(step_inverse(alpha), gran))
    return q, np.asarray(alpha, F32)


# ------------------------------------------------------------------------- ChunkCumsum (mod. 1)
def dt_post(dt_in, dt_softplus: bool) -> np.ndarray:
    """Time step entering the scan: fl32(softplus(dt)) computed in fp64, or dt itself."""
    return fl32(softplus64(dt_in)) if dt_softplus else np.asarray(dt_in, F32)


def _fp64_prefix_exact(v32: np.ndarray) -> bool:
    """True when every fp64 partial sum of each row (last axis) is exact: the row's nonzero
    fp32 terms are multiples of 2^(e_min-24) and partial sums stay below 2^(e_max+log2 n)."""
    n = v32.shape[-1]
    a = np.abs(v32.astype(F64))
    nz = a > 0
    if not nz.any():
        return True
    e = np.frexp(np.where(nz, a, 1.0))[1]
    emax = np.where(nz, e, -100000).max(axis=-1)
    emin = np.where(nz, e, 100000).min(axis=-1)
    has = nz.any(axis=-1)
    need = emax + int(math.ceil(math.log2(max(n, 2)))) - (emin - 24)
    return bool(np.all(~has | (need <= 53)))


def exact_prefix_sum64(v32: np.ndarray) -> np.ndarray:
    """Prefix sums along the last axis, exact and rounded once to fp64."""
    v = np.asarray(v32, F32)
    if _fp64_prefix_exact(v):
        return np.cumsum(v.astype(F64), axis=-1)
    out = np.empty(v.shape, F64)
    flat_in = v.reshape(-1, v.shape[-1]).astype(F64)
    flat_out = out.reshape(-1, v.shape[-1])
    for r in range(flat_in.shape[0]):
        for j in range(flat_in.shape[1]):
            flat_out[r, j] = math.fsum(flat_in[r, :j + 1])
    return out


def chunk_cumsum(dt32_seq, A_h, chunk: int, k: int = 7) -> Dict[str, np.ndarray]:
    """ChunkCumsum for one (batch, head) sequence (Alg. 2 module 1; Eq. 4 LUT; Eq. 9 Q(Decay)).
    dt32_seq (L,) post-softplus fp32.  Returns per chunk (c, Q): dA fp32, cs fp64,
    dec = Decay_state fp32, lut = LUT_state fp32; and q_d (c,) int32."""
    dt = np.asarray(dt32_seq, F32)
    nc = dt.shape[0] // chunk
    dt = dt.reshape(nc, chunk)
    dA = dt * F32(A_h)
    cs = exact_prefix_sum64(dA)
    dec = fl32(np.exp(cs[:, -1:] - cs))
    lut = dt * dec
    qd = np.rint(np.exp(cs[:, -1]) * float(2 ** k)).astype(np.int32)
    return {"dt": dt, "dA": dA, "cs": cs, "dec": dec, "lut": lut, "qd": qd}


# -------------------------------------------------------------- ChunkState (mod. 2, Eq. 7-8)
def _int_matmul(a, b) -> np.ndarray:
    """Integer matrix product through fp64 BLAS (exact: all partial sums are < 2^53)."""
    return np.matmul(np.asarray(a, F64), np.asarray(b, F64)).astype(np.int64)


def requant(acc, mult32) -> np.ndarray:
    """INT32 -> INT8 in registers: clamp(rne(fl32(fl32(acc) * m)), -127, 127)."""
    p = np.asarray(acc).astype(F32) * np.asarray(mult32, F32)
    assert p.dtype == F32
    return np.clip(np.rint(p), -QMAX, QMAX).astype(np.int8)


def multiplier(a1, a2, a3) -> np.ndarray:
    """fl32(a1 * a2 / a3) with the product and quotient formed in fp64."""
    return ((np.asarray(a1, F32).astype(F64) * np.asarray(a2, F32).astype(F64))
            / np.asarray(a3, F32).astype(F64)).astype(F32)


def chunk_state(x_seq, lut, Bq_seq, alpha_xs, alpha_B, alpha_S) -> Dict[str, np.ndarray]:
    """Sparse-aware reformulated ChunkState of one (batch, head) sequence (Eq. 7-8):
    X_scaled = LUT_state o x (fp32), X_q = Q(X_scaled) with per-channel step alpha_xs (P,),
    S32 = X_q^T B_q per chunk (exact int), S_q = requant(S32, a_X a_B / a_S)."""
    nc, Q = lut.shape
    P = x_seq.shape[1]
    x32 = np.asarray(x_seq).astype(F32).reshape(nc, Q, P)
    xs = lut[:, :, None] * x32
    axs = np.broadcast_to(np.asarray(alpha_xs, F32), (P,))
    Xq = quantize(xs, step_inverse(axs)[None, None, :])
    Bq = np.asarray(Bq_seq).reshape(nc, Q, -1)
    S32 = _int_matmul(np.swapaxes(Xq, 1, 2), Bq)                     # (c,P,N)
    mS = multiplier(axs, alpha_B, np.asarray(alpha_S, F32))            # (P,)
    Sq = requant(S32, mS[None, :, None])
    return {"xs": xs, "Xq": Xq.reshape(nc * Q, P), "S32": S32.astype(np.int32), "Sq": Sq,
            "mS": mS}


# -------------------------------------------------------------------- StatePassing (Eq. 9)
def state_pass(Sq, qd, init=None, k: int = 7, shift_round: bool = True):
    """INT8 state passing along the chunk axis (axis 0 of Sq (c, ...), q_d (c,) or (c, ...)
    broadcastable).  Returns (P_in, final): P_in[c] is the state ENTERING chunk c."""
    Sq = np.asarray(Sq)
    nc = Sq.shape[0]
    run = np.zeros(Sq.shape[1:], np.int64) if init is None else np.asarray(init, np.int64).copy()
    pin = np.empty(Sq.shape, np.int8)
    qd = np.asarray(qd, np.int64)
    half = (1 << (k - 1)) if shift_round else 0
    for c in range(nc):
        pin[c] = run
        q = qd[c].reshape(qd[c].shape + (1,) * (run.ndim - np.ndim(qd[c])))
        run = np.clip(Sq[c].astype(np.int64) + ((q * run + half) >> k), -QMAX, QMAX)
    return pin, run.astype(np.int8)


# ------------------------------------------------------------------ ChunkBMM (INT8 CB, Sec 4.2)
def chunk_bmm(Cq_seq, Bq_seq, alpha_C, alpha_B, alpha_CB, chunk: int) -> Dict[str, np.ndarray]:
    """CB32[c,j,i] = C_q[j] . B_q[i] for i <= j, requantized to int8 with m_CB = a_C a_B / a_CB.
    alpha_C is a scalar (per group) or (L,) (per token)."""
    Cq = np.asarray(Cq_seq).reshape(-1, chunk, np.shape(Cq_seq)[-1])
    Bq = np.asarray(Bq_seq).reshape(-1, chunk, np.shape(Bq_seq)[-1])
    causal = np.tril(np.ones((chunk, chunk), bool))
    CB32 = np.where(causal, _int_matmul(Cq, np.swapaxes(Bq, 1, 2)), 0)
    aC = np.asarray(alpha_C, F32)
    mCB = multiplier(aC, alpha_B, alpha_CB)
    if mCB.ndim:
        mCB = mCB.reshape(-1, chunk, 1)
    CBq = np.where(causal, requant(CB32, mCB), 0).astype(np.int8)
    return {"CB32": CB32.astype(np.int32), "CBq": CBq}


# ------------------------------------------------------------------ ChunkScan 1 + 2 and output
def chunk_scan(Cq_seq, pin, CBq, cum, x_seq, alpha_C, alpha_S, alpha_CB, D_h, corr_h,
               out_dtype) -> Dict[str, np.ndarray]:
    """Output of one (batch, head) sequence.  pin (c,P,N) entering states; cum = chunk_cumsum()."""
    nc, Q = cum["cs"].shape
    Cq = np.asarray(Cq_seq).reshape(nc, Q, -1)
    P = x_seq.shape[1]
    cs = cum["cs"]
    aC = np.asarray(alpha_C, F32).astype(F64)
    aC = aC.reshape(nc, Q, 1) if aC.ndim else aC
    Y1 = _int_matmul(Cq, np.swapaxes(np.asarray(pin), 1, 2))          # (c,Q,P)
    y_off = (Y1.astype(F64) * aC * np.asarray(alpha_S, F32).astype(F64)[None, None, :]
             * np.exp(cs)[:, :, None])
    jj, ii = np.meshgrid(np.arange(Q), np.arange(Q), indexing="ij")
    causal = ii <= jj
    seg = np.where(causal[None], cs[:, :, None] - cs[:, None, :], -np.inf)
    W = ((np.asarray(CBq, F64) * float(np.float32(alpha_CB))) * cum["dt"].astype(F64)[:, None, :]
         * np.exp(seg)).astype(np.float16)
    x16 = np.asarray(x_seq).astype(np.float16).reshape(nc, Q, P)
    y_diag = np.matmul(W.astype(F64), x16.astype(F64))
    x32 = np.asarray(x_seq).astype(F32).astype(F64).reshape(nc, Q, P)
    y64 = y_off + y_diag + float(np.float32(D_h)) * x32 + np.asarray(corr_h, F32).astype(F64)
    return {"Y1": Y1.reshape(nc * Q, P).astype(np.int32), "y_off": y_off.reshape(nc * Q, P),
            "y_diag": y_diag.reshape(nc * Q, P), "y64": y64.reshape(nc * Q, P),
            "y": y64.reshape(nc * Q, P).astype(out_dtype)}


# ------------------------------------------------------------------------- whole layer
def scales_for_head(scales: Dict[str, np.ndarray], h: int, g: int, b: int, P: int):
    axs = np.asarray(scales["alpha_Xs"], F32)
    axs_h = np.full(P, axs[h], F32) if axs.ndim == 1 else axs[h]
    aC = np.asarray(scales["alpha_C"], F32)
    aC_bg = aC[b, :, g] if aC.ndim == 3 else aC[g]
    return {"alpha_xs": axs_h, "alpha_B": np.asarray(scales["alpha_B"], F32)[g],
            "alpha_C": aC_bg, "alpha_S": np.asarray(scales["alpha_S"], F32)[h],
            "alpha_CB": np.asarray(scales["alpha_CB"], F32)[g]}


def ssdi8_slab(x_seq, dt32_seq, A_h, Bq_seq, Cq_seq, D_h, corr_h, sc, chunk: int, k: int = 7,
               shift_round: bool = True, init=None, out_dtype=np.float16,
               cbq=None) -> Dict[str, np.ndarray]:
    """Every stage for one (batch, head) sequence.  `sc` from scales_for_head().  `cbq`
    optionally supplies the group's CB_q (it is shared by the heads of a group)."""
    cum = chunk_cumsum(dt32_seq, A_h, chunk, k)
    st = chunk_state(x_seq, cum["lut"], Bq_seq, sc["alpha_xs"], sc["alpha_B"], sc["alpha_S"])
    pin, final_q = state_pass(st["Sq"], cum["qd"], init, k, shift_round)
    if cbq is None:
        cbq = chunk_bmm(Cq_seq, Bq_seq, sc["alpha_C"], sc["alpha_B"], sc["alpha_CB"], chunk)
    scan = chunk_scan(Cq_seq, pin, cbq["CBq"], cum, x_seq, sc["alpha_C"], sc["alpha_S"],
                      sc["alpha_CB"], D_h, corr_h, out_dtype)
    final_state = final_q.astype(F32) * np.asarray(sc["alpha_S"], F32)[:, None]
    out = {"cum": cum, "pin": pin, "final_q": final_q, "final_state": final_state}
    out.update(st)
    out.update(cbq)
    out.update(scan)
    return out


def ssdi8_forward(x, dt_in, A, B, C, D, corr, scales, *, chunk: int, dt_softplus: bool = True,
                  k: int = 7, shift_round: bool = True, init_q=None, out_dtype=None,
                  Bq=None, Cq=None, heads: Optional[Iterable[Tuple[int, int]]] = None,
                  want=("y",)) -> Dict[str, np.ndarray]:
    """Whole quantized SSD layer.  B, C are quantized per group with the static step sizes in
    `scales` unless already-quantized Bq, Cq are passed.  `scales`: alpha_B (G), alpha_C (G) or
    (Bt,L,G) per token, alpha_Xs (H,P) or (H), alpha_S (H,P), alpha_CB (G).
    heads: optional subset of (b, h) pairs; then the result holds per-slab dicts under "slabs".
    want: which full-size global taps to assemble (names as in the module docstring)."""
    Bt, L, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    Q = chunk
    nc = L // Q
    gi = head_group(H, G)
    if out_dtype is None:
        out_dtype = x.dtype
    dt32 = dt_post(dt_in, dt_softplus)
    aC = np.asarray(scales["alpha_C"], F32)
    if Bq is None:
        Bq, _ = quantize_act(B, "group", scales["alpha_B"])
    if Cq is None:
        Cq, _ = quantize_act(C, "token" if aC.ndim == 3 else "group", aC)
    res: Dict[str, np.ndarray] = {"Bq": Bq, "Cq": Cq, "dt": dt32}
    full = heads is None
    pairs = [(b, h) for b in range(Bt) for h in range(H)] if full else list(heads)
    alloc = {
        "y": ((Bt, L, H, P), out_dtype), "y64": ((Bt, L, H, P), F64),
        "Xq": ((Bt, L, H, P), np.int8), "Y1": ((Bt, L, H, P), np.int32),
        "S32": ((Bt, nc, H, P, N), np.int32), "Sq": ((Bt, nc, H, P, N), np.int8),
        "pin": ((Bt, nc, H, P, N), np.int8), "qd": ((Bt, H, nc), np.int32),
        "final_q": ((Bt, H, P, N), np.int8), "final_state": ((Bt, H, P, N), F32),
        "CB32": ((Bt, nc, G, Q, Q), np.int32), "CBq": ((Bt, nc, G, Q, Q), np.int8),
    }
    if full:
        for name in want:
            shp, dty = alloc[name]
            res[name] = np.zeros(shp, dty)
    slabs = {}
    cb_cache: Dict[Tuple[int, int], Dict[str, np.ndarray]] = {}
    for (b, h) in pairs:
        g = int(gi[h])
        sc = scales_for_head(scales, h, g, b, P)
        if (b, g) not in cb_cache:
            cb_cache[(b, g)] = chunk_bmm(Cq[b, :, g], Bq[b, :, g], sc["alpha_C"], sc["alpha_B"],
                                         sc["alpha_CB"], Q)
        init = None if init_q is None else np.asarray(init_q)[b, h]
        s = ssdi8_slab(x[b, :, h], dt32[b, :, h], np.asarray(A, F32)[h], Bq[b, :, g], Cq[b, :, g],
                       np.asarray(D, F32)[h], np.asarray(corr, F32)[h], sc, Q, k, shift_round,
                       init, out_dtype, cbq=cb_cache[(b, g)])
        if not full:
            slabs[(b, h)] = s
            continue
        for name in want:
            if name in ("y", "y64", "Xq", "Y1"):
                res[name][b, :, h] = s[name]
            elif name in ("S32", "Sq", "pin"):
                res[name][b, :, h] = s[name]
            elif name == "qd":
                res[name][b, h] = s["cum"]["qd"]
            elif name in ("final_q", "final_state"):
                res[name][b, h] = s[name]
            elif name in ("CB32", "CBq"):
                res[name][b, :, g] = s[name]
    if not full:
        res["slabs"] = slabs
    return res


# ------------------------------------------------------------------ fragility of fp->int steps
def _ambiguous_fp32(v64: np.ndarray, ulps: float = 4.0) -> np.ndarray:
    """True where rounding v to fp32 could change if v moved by a few fp64 ulps (a result of a
    transcendental function that another correct implementation may round differently)."""
    v = np.asarray(v64, F64)
    eps = ulps * 2.0 ** -52
    return fl32(v * (1 - eps)) != fl32(v * (1 + eps))


def fragile_tokens(dt_in, A_h, chunk: int, dt_softplus: bool, k: int = 7) -> np.ndarray:
    """Per-token flag (L,) for one (batch, head) sequence: True where an fp64 transcendental
    (softplus, or exp in Decay_state / Q(Decay)) lands so close to an fp32 (or integer) rounding
    boundary that a different faithful exp/log1p implementation may round it the other way.  A
    fragile time step poisons the whole chunk (it enters the cumsum)."""
    dt_in = np.asarray(dt_in)
    L = dt_in.shape[0]
    chunk_bad = np.zeros(L // chunk, bool)
    if dt_softplus:
        sp_bad = _ambiguous_fp32(softplus64(dt_in)) & (np.asarray(dt_in, F64) <= 20.0)
        chunk_bad |= sp_bad.reshape(-1, chunk).any(axis=1)
    dt32 = dt_post(dt_in, dt_softplus)
    cum = chunk_cumsum(dt32, A_h, chunk, k)
    tok_bad = _ambiguous_fp32(np.exp(cum["cs"][:, -1:] - cum["cs"])).reshape(-1)
    e = np.exp(cum["cs"][:, -1]) * float(2 ** k)
    chunk_bad |= np.abs(e - np.floor(e) - 0.5) < 1e-9
    return np.repeat(chunk_bad, chunk) | tok_bad
