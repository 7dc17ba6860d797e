"""Pins of the FP16-baseline oracle (oracle/fp16.py) against the fp64 forms of oracle/exact.py:
exact equality where every fp16 / fp32 rounding is exact, the full-reset closed form, and the
fp16 rounding bound on Mamba-shaped inputs."""
import numpy as np
import pytest

from oracle import exact
from oracle import fp16 as ofp

F32 = np.float32


def _tern(rng, shape, density=0.3):
    v = rng.integers(-1, 2, shape)
    return (v * (rng.random(shape) < density)).astype(F32)


@pytest.mark.parametrize("seed", [0, 1])
def test_exactly_representable_case_is_exact(seed):
    # dt = 1, A = 0 (no decay), ternary x/B/C: every fp16 operand and fp32 partial sum is exact
    rng = np.random.default_rng(seed)
    Bt, L, H, P, G, N, Q = 1, 48, 2, 4, 1, 8, 16
    x = _tern(rng, (Bt, L, H, P))
    B = _tern(rng, (Bt, L, G, N))
    C = _tern(rng, (Bt, L, G, N))
    dt = np.ones((Bt, L, H), F32)
    A = np.zeros(H, F32)
    D = np.full(H, 1.0, F32)
    init = rng.integers(-3, 4, (Bt, H, P, N)).astype(F32)
    ref = exact.ssd_chunked(x, dt, A, B, C, D, Q, init.astype(np.float64))
    out = ofp.ssd_fp16_forward(x, dt, A, B, C, D, chunk=Q, dt_softplus=False, init=init)
    assert np.array_equal(out["y64"], ref["y"])
    assert np.array_equal(out["final_state"].astype(np.float64), ref["final_state"])


def test_full_reset_leaves_the_diagonal():
    # A = -1000: every decay underflows to 0, so y_t = (C_t . B_t) dt_t x_t + D x_t
    rng = np.random.default_rng(3)
    Bt, L, H, P, G, N, Q = 1, 32, 2, 4, 1, 8, 16
    x = _tern(rng, (Bt, L, H, P), 0.6)
    B = _tern(rng, (Bt, L, G, N), 0.6)
    C = _tern(rng, (Bt, L, G, N), 0.6)
    dt = np.ones((Bt, L, H), F32)
    A = np.full(H, -1000.0, F32)
    D = np.full(H, 0.5, F32)
    out = ofp.ssd_fp16_forward(x, dt, A, B, C, D, chunk=Q, dt_softplus=False)
    cb = np.einsum("bln,bln->bl", C[:, :, 0], B[:, :, 0])
    expect = cb[:, :, None, None] * x + 0.5 * x
    assert np.array_equal(out["y64"], expect)


def test_fp16_rounding_bound_on_mamba_shaped_inputs():
    # the fp16 operands (X~, W, fp16(P_in)) each carry a relative rounding of at most 2^-11;
    # over the whole layer the output stays within 1e-3 relative L2 of the exact fp64 form
    rng = np.random.default_rng(11)
    Bt, L, H, P, G, N, Q = 2, 128, 4, 16, 2, 32, 32
    x = rng.standard_normal((Bt, L, H, P)).astype(np.float16)
    B = rng.standard_normal((Bt, L, G, N)).astype(np.float16)
    C = rng.standard_normal((Bt, L, G, N)).astype(np.float16)
    dt_raw = rng.normal(-2, 0.5, (Bt, L, H)).astype(F32)
    A = (-np.exp(rng.uniform(0, 2, H))).astype(F32)
    D = rng.normal(1, 0.1, H).astype(F32)
    out = ofp.ssd_fp16_forward(x, dt_raw, A, B, C, D, chunk=Q)
    dt = exact.softplus64(dt_raw).astype(F32)
    ref = exact.ssd_chunked(x, dt, A, B.astype(F32), C.astype(F32), D, Q)
    e = np.linalg.norm(out["y64"] - ref["y"]) / np.linalg.norm(ref["y"])
    assert 1e-6 < e < 1e-3, e
    es = (np.linalg.norm(out["final_state"] - ref["final_state"])
          / np.linalg.norm(ref["final_state"]))
    assert es < 1e-3, es


def test_slab_mode_matches_the_whole_layer():
    rng = np.random.default_rng(5)
    Bt, L, H, P, G, N, Q = 2, 64, 4, 8, 2, 16, 32
    x = rng.standard_normal((Bt, L, H, P)).astype(np.float16)
    B = rng.standard_normal((Bt, L, G, N)).astype(np.float16)
    C = rng.standard_normal((Bt, L, G, N)).astype(np.float16)
    dt_raw = rng.normal(-2, 0.5, (Bt, L, H)).astype(F32)
    A = (-np.exp(rng.uniform(0, 2, H))).astype(F32)
    D = rng.normal(1, 0.1, H).astype(F32)
    full = ofp.ssd_fp16_forward(x, dt_raw, A, B, C, D, chunk=Q)
    part = ofp.ssd_fp16_forward(x, dt_raw, A, B, C, D, chunk=Q, heads=[(1, 3)])
    assert np.array_equal(part["slabs"][(1, 3)]["y64"], full["y64"][1, :, 3])
