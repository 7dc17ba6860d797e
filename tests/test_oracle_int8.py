"""Pins for the quantized SSDi8 oracle (Eq. 1, Sec. 4.2 Eq. 7-9, Eq. 10).

Each pin comes from outside the oracle's own formulas:
  * exact special cases where the quantized path must reproduce the fp64 SSD bit for bit
    (no decay / full reset / zero B or C / power-of-two step sizes);
  * closed forms and hand-worked fixtures (tests/golden);
  * brute force on tiny inputs (explicit loops for the integer contractions and granules);
  * provable error bounds of each fp->int step (|alpha q - v| <= alpha/2 for unclamped values)
    propagated through one contraction;
  * the Eq. 10 invariant (eta = 1 zeroes the per-channel mean error on the calibration draw).
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import calibrate, exact, int8

GOLD = os.path.join(os.path.dirname(__file__), "golden")
F32 = np.float32


# ------------------------------------------------------------------------------ quantizer
def test_quantizer_round_half_even_and_clamp():
    v = np.array([0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 126.5, 127.4, 127.5, 300.0, -300.0, -127.6],
                 F32)
    q = int8.quantize(v, F32(1.0))
    assert q.tolist() == [0, 2, 2, 0, -2, -2, 126, 127, 127, 127, -127, -127]
    assert q.min() >= -127           # -128 is never produced


def test_dynamic_step_is_absmax_over_127_and_zero_granule_is_one():
    rng = np.random.default_rng(0)
    src = rng.standard_normal((2, 3, 4, 5)).astype(F32)
    src[:, :, 2, :] = 0
    q, a = int8.quantize_act(src, "group")
    for k in range(4):
        m = max(abs(float(v)) for v in src[:, :, k, :].ravel())
        expect = F32(1.0) if m == 0 else F32(m) / F32(127)
        assert a[k] == expect
    assert np.all(q[:, :, 2, :] == 0)


@pytest.mark.parametrize("gran", int8.GRANS)
def test_granules_by_brute_force(gran):
    rng = np.random.default_rng(1)
    src = (rng.standard_normal((2, 3, 2, 4)) * 3).astype(F32)
    q, a = int8.quantize_act(src, gran)
    for b in range(2):
        for l in range(3):
            for k in range(2):
                for m in range(4):
                    if gran == "tensor":
                        cell = src
                        alpha = a
                    elif gran == "group":
                        cell = src[:, :, k, :]
                        alpha = a[k]
                    elif gran == "channel":
                        cell = src[:, :, k, m]
                        alpha = a[k, m]
                    else:
                        cell = src[b, l, k, :]
                        alpha = a[b, l, k]
                    amax = max(abs(float(t)) for t in np.ravel(cell))
                    assert alpha == F32(amax) / F32(127)
                    inv = F32(1) / F32(alpha)
                    expect = int(np.clip(np.rint(F32(src[b, l, k, m]) * inv), -127, 127))
                    assert q[b, l, k, m] == expect


def test_quantizer_error_bound():
    rng = np.random.default_rng(2)
    v = (rng.standard_normal(100000) * 7).astype(F32)
    alpha = F32(np.abs(v).max()) / F32(127)
    q = int8.quantize(v, int8.step_inverse(alpha)).astype(np.float64)
    err = np.abs(q * float(alpha) - v.astype(np.float64))
    assert np.all(err <= float(alpha) / 2 * (1 + 1e-6) + np.abs(v) * 2.0 ** -22)


def test_empty_input():
    q, a = int8.quantize_act(np.zeros((0, 4, 1, 8), F32), "group")
    assert q.shape == (0, 4, 1, 8) and a.tolist() == [1.0]


# ------------------------------------------------------------------------------ cumsum
def test_exact_prefix_sum_matches_fsum():
    rng = np.random.default_rng(3)
    v = (-np.exp(rng.uniform(-6, 3, (5, 64)))).astype(F32)
    v[1, ::3] = 0
    s = int8.exact_prefix_sum64(v)
    for r in range(5):
        for j in range(64):
            assert s[r, j] == math.fsum(v[r, :j + 1].astype(np.float64))
    # order independence of exact sums
    assert np.all(np.cumsum(v[:, ::-1].astype(np.float64), axis=1)[:, -1] == s[:, -1])


def test_exact_prefix_sum_wide_span_falls_back_to_fsum():
    v = np.array([[1e20, 1.0, -1e20, 3.0, 1e-20]], F32)
    assert not int8._fp64_prefix_exact(v)
    s = int8.exact_prefix_sum64(v)
    for j in range(5):
        assert s[0, j] == math.fsum(v[0, :j + 1].astype(np.float64))


def test_chunk_cumsum_closed_forms():
    dt = np.full(32, 0.25, F32)
    c = int8.chunk_cumsum(dt, F32(0.0), 16)
    assert np.all(c["dec"] == 1) and np.all(c["lut"] == F32(0.25)) and np.all(c["qd"] == 128)
    c = int8.chunk_cumsum(dt, F32(-2.0), 16)            # dA = -0.5 exactly
    assert np.all(c["cs"][:, -1] == -8.0)
    assert np.all(c["dec"][:, -1] == 1.0)
    assert c["qd"].tolist() == [int(np.rint(np.exp(-8.0) * 128))] * 2 == [0, 0]
    j = np.arange(16)
    assert np.array_equal(c["dec"][0], np.exp(-0.5 * (15 - j)).astype(F32))
    c = int8.chunk_cumsum(np.full(16, 1 / 16, F32), F32(-np.log(2.0)), 16)
    assert c["qd"].tolist() == [64]                     # exp(-ln 2) * 128


# ------------------------------------------------------------------------------ state passing
def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


@pytest.mark.parametrize("mode", ["round", "floor"])
def test_state_pass_hand_fixture(mode):
    g = _load("state_pass_hand.json")
    Sq = np.array(g["S_q"], np.int8).reshape(-1, 1)
    qd = np.array(g["q_d"])
    pin, fin = int8.state_pass(Sq, qd, np.array([g["init"]]), g["k"], mode == "round")
    assert pin[:, 0].tolist() == g["P_in_" + mode]
    assert int(fin[0]) == g["final_" + mode]


def test_state_pass_negative_half():
    pin, fin = int8.state_pass(np.zeros((1, 1), np.int8), np.array([64]), np.array([-3]), 7, True)
    assert int(fin[0]) == -1
    pin, fin = int8.state_pass(np.zeros((1, 1), np.int8), np.array([64]), np.array([-3]), 7, False)
    assert int(fin[0]) == -2


def test_state_pass_identity_decay_is_running_sum_and_zero_decay_copies():
    rng = np.random.default_rng(4)
    Sq = rng.integers(-3, 4, (20, 7, 5)).astype(np.int8)
    pin, fin = int8.state_pass(Sq, np.full(20, 128), None, 7)
    csum = np.concatenate([np.zeros((1, 7, 5), np.int64), np.cumsum(Sq, axis=0, dtype=np.int64)])
    assert np.array_equal(pin, csum[:-1]) and np.array_equal(fin, csum[-1])
    pin, fin = int8.state_pass(Sq, np.zeros(20, int), None, 7)
    assert np.array_equal(pin[1:], Sq[:-1]) and np.array_equal(fin, Sq[-1])


def test_state_pass_saturates_at_127():
    Sq = np.full((10, 3), 100, np.int8)
    Sq[:, 1] = -100
    pin, fin = int8.state_pass(Sq, np.full(10, 128), None, 7)
    assert fin.tolist() == [127, -127, 127]
    assert pin.max() == 127 and pin.min() == -127


def test_state_pass_step_error_bound():
    """Each step is the fp recurrence S + (q_d/2^k) P up to the shift's rounding (<= 1/2)."""
    rng = np.random.default_rng(5)
    Sq = rng.integers(-40, 41, (64, 50)).astype(np.int8)
    qd = rng.integers(0, 129, 64)
    pin, fin = int8.state_pass(Sq, qd, None, 7)
    nxt = np.concatenate([pin[1:], fin[None]]).astype(np.float64)
    fp = Sq + qd[:, None] / 128.0 * pin
    unsat = np.abs(fp) < 126.5
    assert np.all(np.abs(nxt - fp)[unsat] <= 0.5)


# ------------------------------------------------------------------------------ brute force int
def test_integer_contractions_by_brute_force():
    rng = np.random.default_rng(6)
    Q, P, N = 8, 3, 5
    x = rng.standard_normal((2 * Q, P)).astype(F32)
    dt = np.full(2 * Q, 0.5, F32)
    Bq = rng.integers(-127, 128, (2 * Q, N)).astype(np.int8)
    Cq = rng.integers(-127, 128, (2 * Q, N)).astype(np.int8)
    cum = int8.chunk_cumsum(dt, F32(-0.3), Q)
    ax = np.full(P, F32(0.01))
    st = int8.chunk_state(x, cum["lut"], Bq, ax, F32(0.02), np.full(P, F32(3.0)))
    Xq = st["Xq"]
    for c in range(2):
        for p in range(P):
            for n in range(N):
                s = sum(int(Xq[c * Q + j, p]) * int(Bq[c * Q + j, n]) for j in range(Q))
                assert st["S32"][c, p, n] == s
    cb = int8.chunk_bmm(Cq, Bq, F32(0.5), F32(0.25), F32(40.0), Q)
    for c in range(2):
        for j in range(Q):
            for i in range(Q):
                s = sum(int(Cq[c * Q + j, n]) * int(Bq[c * Q + i, n]) for n in range(N))
                assert cb["CB32"][c, j, i] == (s if i <= j else 0)
    pin = rng.integers(-127, 128, (2, P, N)).astype(np.int8)
    scan = int8.chunk_scan(Cq, pin, cb["CBq"], cum, x, F32(0.5), np.ones(P, F32), F32(40.0),
                           F32(0.0), np.zeros(P, F32), np.float32)
    for c in range(2):
        for j in range(Q):
            for p in range(P):
                s = sum(int(Cq[c * Q + j, n]) * int(pin[c, p, n]) for n in range(N))
                assert scan["Y1"][c * Q + j, p] == s


# ------------------------------------------------------------------------------ exact special cases
def _special(seed, L=64, H=2, P=4, G=1, N=8, Q=16, density=0.25, A=0.0, dt=1.0, D=1.0):
    rng = np.random.default_rng(seed)

    def tern(shape):
        v = rng.integers(-1, 2, shape)
        return (v * (rng.random(shape) < density)).astype(F32)
    x = tern((1, L, H, P))
    B = tern((1, L, G, N))
    C = tern((1, L, G, N))
    dtv = np.full((1, L, H), dt, F32)
    Av = np.full(H, A, F32)
    Dv = np.full(H, D, F32)
    return x, dtv, Av, B, C, Dv


def _unit_scales(H, P, G, ax=1.0, ab=1.0, ac=1.0, as_=1.0, acb=1.0):
    return {"alpha_B": np.full(G, ab, F32), "alpha_C": np.full(G, ac, F32),
            "alpha_Xs": np.full((H, P), ax, F32), "alpha_S": np.full((H, P), as_, F32),
            "alpha_CB": np.full(G, acb, F32)}


def _exactness_preconditions(ref, CB_bound=127):
    assert np.abs(ref["states"]).max() <= 127
    assert np.abs(ref["entering"]).max() <= 127 and np.abs(ref["final_state"]).max() <= 127


@pytest.mark.parametrize("Q", [16, 1])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_sc1_no_decay_is_exact(seed, Q):
    # Q = 1 is the recurrent (decode) mode: every token is its own chunk
    x, dt, A, B, C, D = _special(seed)
    H, P, G = 2, 4, 1
    ref = exact.ssd_chunked(x, dt, A, B, C, D, Q)
    _exactness_preconditions(ref)
    out = int8.ssdi8_forward(x, dt, A, B, C, D, np.zeros((H, P), F32), _unit_scales(H, P, G),
                             chunk=Q, dt_softplus=False,
                             want=("y64", "Sq", "pin", "final_q", "CBq", "qd"))
    assert np.array_equal(out["y64"], ref["y"])
    assert np.array_equal(out["Sq"], ref["states"])
    assert np.array_equal(out["pin"], ref["entering"])
    assert np.array_equal(out["final_q"], ref["final_state"])
    assert np.all(out["qd"] == 128)
    CB = np.einsum("bcjn,bcin->bcji", C.reshape(1, -1, Q, 8), B.reshape(1, -1, Q, 8))
    assert np.array_equal(out["CBq"][:, :, 0], np.tril(CB))


@pytest.mark.parametrize("Q", [16, 1])
def test_sc1_with_initial_state_is_exact(Q):
    x, dt, A, B, C, D = _special(7)
    H, P, G, N = 2, 4, 1, 8
    rng = np.random.default_rng(8)
    init = rng.integers(-5, 6, (1, H, P, N)).astype(np.int8)
    ref = exact.ssd_chunked(x, dt, A, B, C, D, Q, init.astype(np.float64))
    _exactness_preconditions(ref)
    out = int8.ssdi8_forward(x, dt, A, B, C, D, np.zeros((H, P), F32), _unit_scales(H, P, G),
                             chunk=Q, dt_softplus=False, init_q=init, want=("y64", "final_q"))
    assert np.array_equal(out["y64"], ref["y"])
    assert np.array_equal(out["final_q"], ref["final_state"])


@pytest.mark.parametrize("seed", [0, 1])
def test_sc2_full_reset_is_exact(seed):
    x, dt, A, B, C, D = _special(seed, A=-1000.0, density=0.6)
    H, P, G, Q = 2, 4, 1, 16
    ref = exact.ssd_chunked(x, dt, A, B, C, D, Q)
    out = int8.ssdi8_forward(x, dt, A, B, C, D, np.zeros((H, P), F32), _unit_scales(H, P, G),
                             chunk=Q, dt_softplus=False, want=("y64", "qd", "Sq", "pin"))
    assert np.all(out["qd"] == 0)
    assert np.array_equal(out["pin"][:, 1:], out["Sq"][:, :-1])
    assert np.array_equal(out["y64"], ref["y"])
    # y_t = (C_t . B_t) x_t + D x_t
    gi = exact.head_group(H, G)
    cb = np.einsum("blhn,blhn->blh", C[:, :, gi], B[:, :, gi])
    assert np.array_equal(out["y64"], cb[..., None] * x + D[None, None, :, None] * x)


@pytest.mark.parametrize("zero", ["B", "C"])
def test_sc3_zero_B_or_C_leaves_skip_plus_correction(zero):
    rng = np.random.default_rng(9)
    Bt, L, H, P, G, N, Q = 2, 32, 4, 8, 2, 16, 16
    x = rng.standard_normal((Bt, L, H, P)).astype(np.float16)
    dt_raw = rng.normal(-2, 0.5, (Bt, L, H)).astype(F32)
    A = (-np.exp(rng.uniform(0, 2, H))).astype(F32)
    B = rng.standard_normal((Bt, L, G, N)).astype(np.float16)
    C = rng.standard_normal((Bt, L, G, N)).astype(np.float16)
    (B if zero == "B" else C)[...] = 0
    D = rng.normal(1, 0.1, H).astype(F32)
    corr = rng.normal(0, 0.1, (H, P)).astype(F32)
    sc = _unit_scales(H, P, G, 0.01, 0.02, 0.03, 0.5, 0.7)
    out = int8.ssdi8_forward(x, dt_raw, A, B, C, D, corr, sc, chunk=Q, want=("y64",))
    expect = (D.astype(np.float64)[None, None, :, None] * x.astype(F32).astype(np.float64)
              + corr.astype(np.float64)[None, None])
    assert np.array_equal(out["y64"], expect)


@pytest.mark.parametrize("dtv", [1.0, 0.5])
def test_sc4_power_of_two_steps_are_exact(dtv):
    rng = np.random.default_rng(10)
    L, H, P, G, N, Q = 48, 2, 4, 1, 8, 16
    kx = rng.integers(-3, 4, (1, L, H, P)) * (rng.random((1, L, H, P)) < 0.3)
    kb = rng.integers(-2, 3, (1, L, G, N)) * (rng.random((1, L, G, N)) < 0.3)
    kc = rng.integers(-2, 3, (1, L, G, N)) * (rng.random((1, L, G, N)) < 0.3)
    ax = 2.0 ** -3 * dtv
    x = (kx * 2.0 ** -3).astype(F32)
    B = (kb * 2.0 ** -2).astype(F32)
    C = (kc * 2.0 ** -1).astype(F32)
    dt = np.full((1, L, H), dtv, F32)
    A = np.zeros(H, F32)
    D = np.full(H, 0.75, F32)
    ab, ac = 2.0 ** -2, 2.0 ** -1
    sc = _unit_scales(H, P, G, ax, ab, ac, ax * ab, ac * ab)
    ref = exact.ssd_chunked(x, dt, A, B, C, D, Q)
    assert np.abs(ref["states"] / (ax * ab)).max() <= 127
    assert np.abs(ref["entering"] / (ax * ab)).max() <= 127
    out = int8.ssdi8_forward(x, dt, A, B, C, D, np.zeros((H, P), F32), sc, chunk=Q,
                             dt_softplus=False, want=("y64", "Sq", "final_state"))
    assert np.array_equal(out["y64"], ref["y"])
    assert np.array_equal(out["Sq"] * (ax * ab), ref["states"])
    assert np.array_equal(out["final_state"].astype(np.float64), ref["final_state"])


def test_hand_fixture_through_quantized_path():
    g = _load("ssd_hand.json")
    L = len(g["x"])
    x = np.array(g["x"], F32).reshape(1, L, 1, 1)
    B = np.array(g["B"], F32).reshape(1, L, 1, 1)
    C = np.array(g["C"], F32).reshape(1, L, 1, 1)
    out = int8.ssdi8_forward(x, np.ones((1, L, 1), F32), np.zeros(1, F32), B, C,
                             np.array([g["D"]], F32), np.zeros((1, 1), F32),
                             _unit_scales(1, 1, 1), chunk=g["chunk"], dt_softplus=False,
                             want=("y64", "Sq", "pin", "final_q"))
    assert out["y64"].ravel().tolist() == g["y"]
    assert out["Sq"].ravel().tolist() == g["local_states"]
    assert out["pin"].ravel().tolist() == g["entering"]
    assert int(out["final_q"].ravel()[0]) == g["final"]


# ------------------------------------------------------------------------------ stage error bounds
def _random_layer(seed=11, Bt=1, L=64, H=3, P=8, G=1, N=16, Q=32):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((Bt, L, H, P)).astype(np.float16)
    dt_raw = rng.normal(-2, 0.5, (Bt, L, H)).astype(F32)
    A = (-np.exp(rng.uniform(0, np.log(16), H))).astype(F32)
    B = rng.standard_normal((Bt, L, G, N)).astype(np.float16)
    C = rng.standard_normal((Bt, L, G, N)).astype(np.float16)
    D = rng.normal(1, 0.1, H).astype(F32)
    return x, dt_raw, A, B, C, D, Q


def test_chunk_state_within_quantization_bound():
    x, dt_raw, A, B, C, D, Q = _random_layer()
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q)
    dt32 = int8.dt_post(dt_raw, True)
    Bq, _ = int8.quantize_act(B, "group", sc["alpha_B"])
    aB = float(sc["alpha_B"][0])
    for h in range(3):
        cum = int8.chunk_cumsum(dt32[0, :, h], A[h], Q)
        st = int8.chunk_state(x[0, :, h], cum["lut"], Bq[0, :, 0], sc["alpha_Xs"][h], aB,
                              sc["alpha_S"][h])
        ax = sc["alpha_Xs"][h].astype(np.float64)
        xs = st["xs"].astype(np.float64)                                  # (c,Q,P)
        Bv = B[0, :, 0].astype(np.float64).reshape(-1, Q, 16)
        exact_s = np.matmul(np.swapaxes(xs, 1, 2), Bv)
        approx = st["S32"] * ax[None, :, None] * aB
        ex = ax[None, None, :] / 2 * (1 + 1e-6) + np.abs(xs) * 2.0 ** -22
        eb = aB / 2 * (1 + 1e-6) + np.abs(Bv) * 2.0 ** -22
        bound = (np.matmul(np.swapaxes(np.abs(xs), 1, 2), eb)
                 + np.matmul(np.swapaxes(ex, 1, 2), np.abs(Bv))
                 + np.matmul(np.swapaxes(ex, 1, 2), np.broadcast_to(eb, Bv.shape)))
        assert np.all(np.abs(approx - exact_s) <= bound)
        # requantization of the accumulator: within half a state step unless saturated
        aS = sc["alpha_S"][h].astype(np.float64)[None, :, None]
        unsat = np.abs(st["Sq"]) < 127
        err = np.abs(st["Sq"] * aS - approx)
        assert np.all(err[unsat] <= (aS / 2 * (1 + 1e-5) + np.abs(approx) * 2.0 ** -21)[unsat])


def test_chunk_bmm_within_quantization_bound():
    x, dt_raw, A, B, C, D, Q = _random_layer(12)
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q)
    Bq, _ = int8.quantize_act(B, "group", sc["alpha_B"])
    Cq, _ = int8.quantize_act(C, "group", sc["alpha_C"])
    aB, aC, aCB = (float(sc[k][0]) for k in ("alpha_B", "alpha_C", "alpha_CB"))
    cb = int8.chunk_bmm(Cq[0, :, 0], Bq[0, :, 0], aC, aB, aCB, Q)
    Bv = B[0, :, 0].astype(np.float64).reshape(-1, Q, 16)
    Cv = C[0, :, 0].astype(np.float64).reshape(-1, Q, 16)
    exact_cb = np.tril(np.matmul(Cv, np.swapaxes(Bv, 1, 2)))
    approx = cb["CB32"] * aC * aB
    ec = aC / 2 * (1 + 1e-6) + np.abs(Cv) * 2.0 ** -22
    eb = aB / 2 * (1 + 1e-6) + np.abs(Bv) * 2.0 ** -22
    bound = np.tril(np.matmul(np.abs(Cv), np.swapaxes(eb, 1, 2))
                    + np.matmul(ec, np.swapaxes(np.abs(Bv), 1, 2))
                    + np.matmul(ec, np.swapaxes(eb, 1, 2)))
    assert np.all(np.abs(approx - exact_cb) <= bound)
    unsat = np.abs(cb["CBq"]) < 127
    err = np.abs(cb["CBq"] * aCB - approx)
    assert np.all(err[unsat] <= (aCB / 2 * (1 + 1e-5) + np.abs(approx) * 2.0 ** -21)[unsat])


def test_chunk_scan_terms_closed_form_and_fp16_bound():
    x, dt_raw, A, B, C, D, Q = _random_layer(13)
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q)
    out = int8.ssdi8_forward(x, dt_raw, A, B, C, D, sc["corr"], sc, chunk=Q, heads=[(0, 1)])
    s = out["slabs"][(0, 1)]
    cs = s["cum"]["cs"]
    # ChunkScan1 closed form from its own integer product
    aC, aS = float(sc["alpha_C"][0]), sc["alpha_S"][1].astype(np.float64)
    expect_off = (s["Y1"].reshape(-1, Q, 8) * aC * aS[None, None, :] * np.exp(cs)[:, :, None])
    assert np.allclose(s["y_off"].reshape(-1, Q, 8), expect_off, rtol=1e-14, atol=0)
    # ChunkScan2 against unrounded fp64 weights: two fp16 roundings per term at most
    aCB = float(sc["alpha_CB"][0])
    dt = s["cum"]["dt"].astype(np.float64)
    jj, ii = np.meshgrid(np.arange(Q), np.arange(Q), indexing="ij")
    seg = np.where(ii <= jj, cs[:, :, None] - cs[:, None, :], -np.inf)
    Wex = s["CBq"] * aCB * dt[:, None, :] * np.exp(seg)
    xv = x[0, :, 1].astype(np.float64).reshape(-1, Q, 8)
    ydx = np.matmul(Wex, xv)
    bound = np.matmul(np.abs(Wex) * 2.0 ** -11 + 2.0 ** -24, np.abs(xv)) * (1 + 1e-9)
    assert np.all(np.abs(s["y_diag"].reshape(-1, Q, 8) - ydx) <= bound + 1e-12)


def test_mean_correction_eta_one_zeroes_channel_mean_error():
    """Eq. 10: with eta = 1 the correction equals the per-channel mean error on the draw it was
    estimated from, so the corrected output has zero mean error per channel."""
    x, dt_raw, A, B, C, D, Q = _random_layer(14, Bt=2)
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q, eta=1.0)
    out = int8.ssdi8_forward(x, dt_raw, A, B, C, D, sc["corr"], sc, chunk=Q, want=("y64",))
    dt32 = int8.dt_post(dt_raw, True).astype(np.float64)
    ref = exact.ssd_chunked(x.astype(np.float64), dt32, A.astype(np.float64), B, C, D, Q)
    resid = (ref["y"] - out["y64"]).mean(axis=(0, 1))
    # corr is stored in fp32: the residual is its fp32 rounding error
    assert np.all(np.abs(resid) <= np.abs(sc["corr"]) * 2.0 ** -23 + 1e-12)
    out0 = int8.ssdi8_forward(x, dt_raw, A, B, C, D, np.zeros_like(sc["corr"]), sc, chunk=Q,
                              want=("y64",))
    assert np.abs((ref["y"] - out0["y64"]).mean(axis=(0, 1))).max() > 100 * np.abs(resid).max()


def test_calibrated_state_scale_rarely_saturates_on_its_own_draw():
    x, dt_raw, A, B, C, D, Q = _random_layer(15, Bt=2, L=128)
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q)
    out = int8.ssdi8_forward(x, dt_raw, A, B, C, D, sc["corr"], sc, chunk=Q,
                             want=("Sq", "pin", "CBq"))
    for name in ("Sq", "pin", "CBq"):
        assert np.mean(np.abs(out[name]) == 127) < 0.01, name


def test_quantized_layer_tracks_fp64_layer():
    """End-to-end the quantized layer stays close to the fp64 SSD on outlier-free data (a wrong
    index, sign or scale anywhere gives an O(1) error)."""
    x, dt_raw, A, B, C, D, Q = _random_layer(16, Bt=2, L=128)
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q)
    out = int8.ssdi8_forward(x, dt_raw, A, B, C, D, sc["corr"], sc, chunk=Q, want=("y64",))
    dt32 = int8.dt_post(dt_raw, True).astype(np.float64)
    ref = exact.ssd_chunked(x.astype(np.float64), dt32, A.astype(np.float64), B, C, D, Q)
    rel = np.linalg.norm(out["y64"] - ref["y"]) / np.linalg.norm(ref["y"])
    assert rel < 0.03


def test_per_token_C_scales_factor_out():
    """Per-token C steps (one per (b,l,g)) factor out of C.B^T rows and of ChunkScan1; with
    every token's step equal to the group step the result is identical to per-group."""
    x, dt_raw, A, B, C, D, Q = _random_layer(17)
    sc = calibrate.calibrate(x, dt_raw, A, B, C, D, chunk=Q)
    tok = dict(sc)
    tok["alpha_C"] = np.broadcast_to(sc["alpha_C"][None, None, :], (1, 64, 1)).copy()
    a = int8.ssdi8_forward(x, dt_raw, A, B, C, D, sc["corr"], sc, chunk=Q, want=("y64",))
    b = int8.ssdi8_forward(x, dt_raw, A, B, C, D, sc["corr"], tok, chunk=Q, want=("y64",))
    assert np.array_equal(a["y64"], b["y64"])


def test_fragile_tokens_are_rare():
    rng = np.random.default_rng(18)
    raw = rng.normal(-2, 0.5, 4096).astype(F32)
    bad = int8.fragile_tokens(raw, F32(-3.0), 256, True)
    assert bad.mean() < 0.01


def test_decode_steps_chain_through_the_int8_state():
    """The recurrent mode (a chunk of one token, Sec. 4.2 state passing with Eq. 9 per token):
    T single-token calls chained through the final int8 state equal one call over T tokens
    with chunk 1, stage by stage."""
    rng = np.random.default_rng(21)
    Bt, T, H, P, G, N = 2, 6, 4, 8, 2, 16
    x = rng.standard_normal((Bt, T, H, P)).astype(np.float16)
    dt_raw = rng.normal(-2, 0.5, (Bt, T, H)).astype(F32)
    A = (-np.exp(rng.uniform(0, 2, H))).astype(F32)
    B = rng.standard_normal((Bt, T, G, N)).astype(np.float16)
    C = rng.standard_normal((Bt, T, G, N)).astype(np.float16)
    D = rng.normal(1, 0.1, H).astype(F32)
    corr = rng.normal(0, 0.1, (H, P)).astype(F32)
    sc = _unit_scales(H, P, G, 0.02, 0.03, 0.03, 0.05, 0.1)
    init = rng.integers(-60, 61, (Bt, H, P, N)).astype(np.int8)
    whole = int8.ssdi8_forward(x, dt_raw, A, B, C, D, corr, sc, chunk=1, init_q=init,
                               want=("y64", "final_q", "pin"))
    state = init
    for t in range(T):
        one = int8.ssdi8_forward(x[:, t:t + 1], dt_raw[:, t:t + 1], A, B[:, t:t + 1],
                                 C[:, t:t + 1], D, corr, sc, chunk=1, init_q=state,
                                 want=("y64", "final_q", "pin"))
        assert np.array_equal(one["pin"][:, 0], whole["pin"][:, t])
        assert np.array_equal(one["y64"][:, 0], whole["y64"][:, t])
        state = one["final_q"]
    assert np.array_equal(state, whole["final_q"])
    assert np.abs(whole["pin"].astype(int)).max() > 20        # the state is exercised
