"""GPU parity of the single-token decode step (ssdi8_decode_step) against the oracle run with a
chunk of one token: every new int8 state bit-exact, y within the stated tolerance, over chains
of steps, after a chunked prefill, and across the dtype / scale-granularity variants."""
import dataclasses

import numpy as np
import pytest

from helpers import assert_close, assert_equal, calibration, dev, say
from oracle import int8 as oq
from paper_2608_21952_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    assert _t.cuda.is_available(), "GPU tests need a GPU"
    return _t


@pytest.fixture(scope="module")
def ssdi8(torch):
    from paper_2608_21952_amd import ssdi8 as _s
    _s.lib()
    return _s


def _cfg(name="decode-g4", **kw):
    base = dict(name=name, batch=2, seqlen=512, nheads=16, ngroups=4, xs_per_head=False)
    base.update(kw)
    return dataclasses.replace(synth.CONFIGS["mamba2-8b-g8"], **base)


def _gpu_steps(torch, ssdi8, inp, sc, init, T, *, x_dtype=None, y_dtype=None, c_tok=None,
               with_skip=True, state_f32=False):
    """T decode steps on the GPU from `init`; returns per-step y and states (numpy)."""
    Bt, L, H, P = inp["x"].shape
    G = inp["B"].shape[2]
    f = lambda v: dev(np.asarray(v, np.float32), torch)
    A, D, corr = f(inp["A"]), f(inp["D"]), f(sc["corr"])
    aB, aS, aCB = f(sc["alpha_B"]), f(sc["alpha_S"]), f(sc["alpha_CB"])
    aX = f(sc["alpha_Xs"])                           # (H, P), or (H) per head
    state = dev(init, torch)
    ys, states, fstates = [], [], []
    for t in range(T):
        x = inp["x"][:, t]
        if x_dtype is not None:
            x = x.astype(x_dtype)
        xt = dev(x, torch)
        dtt = f(inp["dt_raw"][:, t])
        Bt_ = dev(inp["B"][:, t:t + 1], torch)
        Ct_ = dev(inp["C"][:, t:t + 1], torch)
        Bq = ssdi8.quantize_act(Bt_, "group", aB)[0].reshape(Bt, G, -1)
        if c_tok is None:
            aC = f(sc["alpha_C"])
            Cq = ssdi8.quantize_act(Ct_, "group", aC)[0].reshape(Bt, G, -1)
        else:
            aC = f(c_tok[:, t])                      # (Bt, G) per-token C steps
            Cq = ssdi8.quantize_act(Ct_, "token", f(c_tok[:, t:t + 1]))[0].reshape(Bt, G, -1)
        out = ssdi8.decode_step(xt, dtt, A, Bq, Cq, aB, aC, aX, aS, aCB, state,
                                D=D if with_skip else None, corr=corr if with_skip else None,
                                y_dtype=y_dtype, state_f32=state_f32)
        ys.append(out["y"].float().cpu().numpy())
        states.append(state.cpu().numpy().copy())
        if state_f32:
            fstates.append(out["state"].cpu().numpy())
    return np.stack(ys, 1), states, fstates


def _oracle_steps(inp, sc, init, T, *, x_dtype=None, c_tok=None, with_skip=True):
    x = inp["x"][:, :T]
    if x_dtype is not None:
        x = x.astype(x_dtype)
    scales = dict(sc)
    if c_tok is not None:
        scales["alpha_C"] = c_tok[:, :T]
    H, P = x.shape[2], x.shape[3]
    D = inp["D"] if with_skip else np.zeros(H, np.float32)
    corr = sc["corr"] if with_skip else np.zeros((H, P), np.float32)
    return oq.ssdi8_forward(x, inp["dt_raw"][:, :T], inp["A"], inp["B"][:, :T], inp["C"][:, :T],
                            D, corr, scales, chunk=1, init_q=init,
                            want=("y64", "pin", "final_q", "final_state"))


def _check(ys, states, ref, T, what):
    for t in range(T):
        nxt = ref["pin"][:, t + 1] if t + 1 < T else ref["final_q"]
        assert_equal(states[t], nxt, f"{what}: state after token {t}")
    assert_close(ys, ref["y64"], f"{what}: y over {T} tokens")


def test_decode_chain_matches_oracle(torch, ssdi8):
    cfg = _cfg()
    say(f"decode chain: B={cfg.batch} H={cfg.nheads} G={cfg.ngroups}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    rng = np.random.default_rng(5)
    init = rng.integers(-100, 101, (cfg.batch, cfg.nheads, 64, 128)).astype(np.int8)
    T = 12
    ys, states, fst = _gpu_steps(torch, ssdi8, inp, sc, init, T, state_f32=True)
    ref = _oracle_steps(inp, sc, init, T)
    _check(ys, states, ref, T, "fp16")
    assert_close(fst[-1], ref["final_state"], "fp32 state")


def test_decode_variants(torch, ssdi8):
    """fp32 x and y, per-token C steps, one X_scaled step per head, no skip / correction."""
    cfg = _cfg("decode-var", nheads=8, ngroups=2, xs_per_head=True)
    inp = synth.draw(cfg, 3)
    sc = calibration(cfg)
    rng = np.random.default_rng(6)
    init = rng.integers(-127, 128, (cfg.batch, cfg.nheads, 64, 128)).astype(np.int8)
    T = 5
    C32 = np.asarray(inp["C"][:, :T], np.float32)
    c_tok = np.maximum(np.abs(C32).max(axis=3) / 127.0, 1e-6).astype(np.float32)  # (Bt,T,G)
    ys, states, _ = _gpu_steps(torch, ssdi8, inp, sc, init, T, x_dtype=np.float32,
                               y_dtype=torch.float32, c_tok=c_tok, with_skip=False)
    assert sc["alpha_Xs"].ndim == 1
    ref = _oracle_steps(inp, sc, init, T, x_dtype=np.float32, c_tok=c_tok, with_skip=False)
    _check(ys, states, ref, T, "fp32 / per-token C / per-head X")


def test_prefill_then_decode(torch, ssdi8):
    """The int8 state left by a chunked prefill continues token by token."""
    cfg = _cfg("decode-prefill", nheads=8, ngroups=2)
    inp = synth.draw(cfg, 4)
    sc = calibration(cfg)
    Lp = 256
    f = lambda v: dev(np.asarray(v, np.float32), torch)
    Bq = ssdi8.quantize_act(dev(inp["B"][:, :Lp], torch), "group", f(sc["alpha_B"]))[0]
    Cq = ssdi8.quantize_act(dev(inp["C"][:, :Lp], torch), "group", f(sc["alpha_C"]))[0]
    pre = ssdi8.ssd_chunk_scan(dev(inp["x"][:, :Lp], torch), f(inp["dt_raw"][:, :Lp]),
                               f(inp["A"]), Bq, Cq, f(sc["alpha_B"]), f(sc["alpha_C"]),
                               f(sc["alpha_Xs"]), f(sc["alpha_S"]), f(sc["alpha_CB"]),
                               D=f(inp["D"]), corr=f(sc["corr"]))
    ref_pre = oq.ssdi8_forward(inp["x"][:, :Lp], inp["dt_raw"][:, :Lp], inp["A"],
                               inp["B"][:, :Lp], inp["C"][:, :Lp], inp["D"], sc["corr"], sc,
                               chunk=256, want=("final_q",))
    state0 = pre["final_state_q"].cpu().numpy()
    assert_equal(state0, ref_pre["final_q"], "prefill final state")
    tail = {k: (v[:, Lp:] if k in ("x", "dt_raw", "B", "C") else v) for k, v in inp.items()}
    T = 3
    ys, states, _ = _gpu_steps(torch, ssdi8, tail, sc, state0, T)
    ref = _oracle_steps(tail, sc, ref_pre["final_q"], T)
    _check(ys, states, ref, T, "after prefill")


def test_decode_empty_batch(torch, ssdi8):
    z = lambda *s: torch.zeros(s, dtype=torch.float32, device="cuda")
    st = torch.zeros((0, 4, 64, 128), dtype=torch.int8, device="cuda")
    q = torch.zeros((0, 2, 128), dtype=torch.int8, device="cuda")
    out = ssdi8.decode_step(torch.zeros((0, 4, 64), dtype=torch.float16, device="cuda"),
                            z(0, 4), z(4), q, q, z(2), z(2), z(4, 64), z(4, 64), z(2), st)
    assert out["y"].shape == (0, 4, 64)
