"""Pins of the oracle's static calibration (Sec. 5 setup: symmetric static steps fixed offline;
Eq. 1 step = absmax / 127; Eq. 7 X_scaled; Eq. 4 / Eq. 8 states; CB per group, causal entries).

Every step size is recomputed here from its definition with explicit scalar loops that share no
code with `oracle.calibrate`:
  alpha_B, alpha_C   absmax over (b, l, n) of the fp32 values of B / C in group g, / 127
  alpha_Xs           absmax over (b, t) of X_scaled = fl32(LUT_state * x), per (h, p) or per h,
                     with LUT_state_j = fl32(dt_j * fl32(exp(sum of dA over the rest of the
                     chunk))) and the in-chunk sums taken exactly (math.fsum)
  alpha_S            absmax over (b, c, n) of the unquantized states, both the chunk-local ones
                     (the recurrence restarted from zero at each chunk start, Eq. 4) and the
                     states passed out of each chunk (the recurrence run through), / 127
  alpha_CB           absmax over (b, c) and the causal entries i <= j of C_j . B_i, / 127
The states come from the token-by-token recurrence h = exp(dt A) h + dt x B^T, not from the
chunked form the oracle uses, so a wrong decay, a dropped term or a missing passed state shows.
The draws are built so that the passed states exceed the chunk-local ones and an acausal entry of
C.B^T exceeds every causal one: a step taken over the wrong set then differs by far more than
the rounding between the two computations (relative 1e-6 is allowed for the fp64 ones).
"""
import math

import numpy as np
import pytest

from oracle import calibrate

F32 = np.float32


def _layer(seed, Bt=2, L=160, H=4, P=4, G=2, N=5, Q=16):
    """A tiny layer with slow decay (the passed states grow past the chunk-local ones) and one
    planted acausal C.B^T outlier per group: C at the first token of a chunk and B at its last
    token, so that their product sits at (j, i) = (0, Q - 1), above the diagonal.  x is zero at
    that last token, so the B outlier does not reach the states."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((Bt, L, H, P))
    x[:, Q - 1] = 0.0
    x = x.astype(np.float16)
    dt_raw = rng.normal(-2.0, 0.5, (Bt, L, H)).astype(F32)
    A = (-np.exp(rng.uniform(-6.0, -4.0, H))).astype(F32)
    B = rng.standard_normal((Bt, L, G, N))
    C = rng.standard_normal((Bt, L, G, N))
    B[:, Q - 1, :, :] *= 9.0          # last token of chunk 0
    C[:, 0, :, :] *= 9.0              # first token of chunk 0
    D = rng.normal(1.0, 0.1, H).astype(F32)
    return (x, dt_raw, A, B.astype(np.float16), C.astype(np.float16), D, Q)


def _step(absmax: float) -> F32:
    a = F32(F32(absmax) / F32(127.0))
    return F32(1.0) if a == 0 else a


def _softplus32(v: float) -> F32:
    """fl32 of softplus(v) = log(1 + exp(v)), v itself above 20."""
    v = float(v)
    return F32(v if v > 20.0 else math.log1p(math.exp(v)))


def _brute_scales(x, dt_raw, A, B, C, Q, xs_per_head=False):
    Bt, L, H, P = x.shape
    G, N = B.shape[2], B.shape[3]
    hpg = H // G
    nc = L // Q
    B32, C32, x32 = B.astype(F32), C.astype(F32), x.astype(F32)
    out = {}
    out["alpha_B"] = np.array([_step(max(abs(float(B32[b, l, g, n])) for b in range(Bt)
                                         for l in range(L) for n in range(N)))
                               for g in range(G)], F32)
    out["alpha_C"] = np.array([_step(max(abs(float(C32[b, l, g, n])) for b in range(Bt)
                                         for l in range(L) for n in range(N)))
                               for g in range(G)], F32)
    xs_max = np.zeros((H, P))
    s_local = np.zeros((H, P))
    s_passed = np.zeros((H, P))
    for b in range(Bt):
        for h in range(H):
            g = h // hpg
            dt = [_softplus32(dt_raw[b, t, h]) for t in range(L)]
            # X_scaled (Eq. 7): LUT_state from the exact in-chunk sums of fl32(dt A)
            for c in range(nc):
                dA = [float(F32(dt[c * Q + j] * A[h])) for j in range(Q)]
                for j in range(Q):
                    rest = math.fsum(dA[:Q]) - math.fsum(dA[:j + 1])
                    dec = F32(math.exp(rest))
                    lut = F32(dt[c * Q + j] * dec)
                    for p in range(P):
                        v = abs(float(F32(lut * x32[b, c * Q + j, h, p])))
                        xs_max[h, p] = max(xs_max[h, p], v)
            # states (Eq. 4 chunk-local; passed = the recurrence run through every chunk)
            run = np.zeros((P, N))
            for c in range(nc):
                loc = np.zeros((P, N))
                for j in range(Q):
                    t = c * Q + j
                    a = math.exp(float(dt[t]) * float(A[h]))
                    u = float(dt[t]) * np.outer(x32[b, t, h].astype(np.float64),
                                                B32[b, t, g].astype(np.float64))
                    loc = a * loc + u
                    run = a * run + u
                s_local[h] = np.maximum(s_local[h], np.abs(loc).max(axis=1))
                s_passed[h] = np.maximum(s_passed[h], np.abs(run).max(axis=1))
    if xs_per_head:
        out["alpha_Xs"] = np.array([_step(xs_max[h].max()) for h in range(H)], F32)
    else:
        out["alpha_Xs"] = np.array([[_step(xs_max[h, p]) for p in range(P)] for h in range(H)],
                                   F32)
    s_all = np.maximum(s_local, s_passed)
    out["alpha_S"] = np.array([[_step(s_all[h, p]) for p in range(P)] for h in range(H)], F32)
    cb_causal = np.zeros(G)
    cb_any = np.zeros(G)
    for b in range(Bt):
        for g in range(G):
            for c in range(nc):
                for j in range(Q):
                    cj = C32[b, c * Q + j, g].astype(np.float64)
                    for i in range(Q):
                        v = abs(math.fsum(cj * B32[b, c * Q + i, g].astype(np.float64)))
                        cb_any[g] = max(cb_any[g], v)
                        if i <= j:
                            cb_causal[g] = max(cb_causal[g], v)
    out["alpha_CB"] = np.array([_step(v) for v in cb_causal], F32)
    return out, {"s_local": s_local, "s_passed": s_passed, "cb_causal": cb_causal,
                 "cb_any": cb_any, "xs_max": xs_max}


@pytest.mark.parametrize("xs_per_head", [False, True])
def test_calibrated_steps_match_their_definitions(xs_per_head):
    x, dt_raw, A, B, C, D, Q = _layer(31)
    ref, raw = _brute_scales(x, dt_raw, A, B, C, Q, xs_per_head=xs_per_head)
    # the draw separates the candidate definitions clearly
    assert np.mean(raw["s_passed"] > 1.2 * raw["s_local"]) > 0.75, "passed states must dominate"
    assert np.all(raw["cb_any"] > 1.5 * raw["cb_causal"]), "an acausal C.B^T entry must dominate"
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q, xs_per_head=xs_per_head)
    # quantities the quantizers see in fp32: identical
    for k in ("alpha_B", "alpha_C", "alpha_Xs"):
        assert sc[k].dtype == F32 and sc[k].shape == ref[k].shape, k
        assert np.array_equal(sc[k], ref[k]), (k, sc[k], ref[k])
    # fp64 statistics (states, C.B^T) from another summation order: to 1e-6 relative
    for k in ("alpha_S", "alpha_CB"):
        assert sc[k].dtype == F32 and sc[k].shape == ref[k].shape, k
        np.testing.assert_allclose(sc[k], ref[k], rtol=1e-6, atol=0, err_msg=k)


def test_state_step_covers_the_passed_states_not_only_the_chunk_local_ones():
    """With a fast decay the chunk-local states dominate instead; the step follows whichever
    of the two sets holds the larger magnitude, channel by channel."""
    x, dt_raw, A, B, C, D, Q = _layer(32)
    A = (-np.exp(np.random.default_rng(5).uniform(1.0, 2.0, A.shape[0]))).astype(F32)
    ref, raw = _brute_scales(x, dt_raw, A, B, C, Q)
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q)
    np.testing.assert_allclose(sc["alpha_S"], ref["alpha_S"], rtol=1e-6, atol=0)
    np.testing.assert_allclose(sc["alpha_S"],
                               (np.maximum(raw["s_local"], raw["s_passed"]) / 127).astype(F32),
                               rtol=1e-6, atol=0)


def test_all_zero_granules_get_a_unit_step():
    """Eq. 1 with absmax = 0 would divide by zero; the reading gives such a granule step 1:
    B of group 0, C of group 1, every channel of head 0 (x = 0 there, so its X_scaled and its
    states are zero) and the C.B^T of both groups (one of B, C is zero in each)."""
    x, dt_raw, A, B, C, D, Q = _layer(33)
    B = B.copy()
    C = C.copy()
    x = x.copy()
    B[:, :, 0] = 0
    C[:, :, 1] = 0
    x[:, :, 0] = 0
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q)
    assert sc["alpha_B"][0] == 1 and sc["alpha_C"][1] == 1
    assert np.all(sc["alpha_Xs"][0] == 1) and np.all(sc["alpha_S"][0] == 1)
    assert np.all(sc["alpha_CB"] == 1)
    assert sc["alpha_B"][1] != 1 and sc["alpha_C"][0] != 1 and np.all(sc["alpha_Xs"][1:] != 1)
