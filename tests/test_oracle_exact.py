"""Pins for the fp64 SSD forms of the oracle (Sec. 4.1 duality, Alg. 2 chunking).

The three forms are written independently (a time loop, a dense masked matrix, and the five
chunked modules); agreement on random tiny inputs pins the chunk-boundary conventions (which
state Scan1 reads, the dt factor placement in LUT_scan1/LUT_scan2, the causal mask)."""
import numpy as np
import pytest

from oracle import exact


def _rand(seed, Bt=2, L=24, H=4, P=3, G=2, N=5):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((Bt, L, H, P))
    dt = np.log1p(np.exp(rng.normal(-1.0, 0.7, (Bt, L, H))))
    A = -np.exp(rng.uniform(-1.0, 1.5, H))
    B = rng.standard_normal((Bt, L, G, N))
    C = rng.standard_normal((Bt, L, G, N))
    D = rng.normal(1.0, 0.1, H)
    init = rng.standard_normal((Bt, H, P, N))
    return x, dt, A, B, C, D, init


def _rel(a, b):
    return np.abs(a - b).max() / max(np.abs(b).max(), 1e-300)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_quadratic_equals_recurrence(seed):
    x, dt, A, B, C, D, init = _rand(seed)
    r = exact.ssd_recurrence(x, dt, A, B, C, D, init)
    q = exact.ssd_quadratic(x, dt, A, B, C, D, init)
    assert _rel(q["y"], r["y"]) < 1e-12


@pytest.mark.parametrize("chunk", [1, 2, 3, 4, 6, 8, 12, 24])
def test_chunked_equals_recurrence_any_chunk(chunk):
    x, dt, A, B, C, D, init = _rand(5)
    r = exact.ssd_recurrence(x, dt, A, B, C, D, init)
    c = exact.ssd_chunked(x, dt, A, B, C, D, chunk, init)
    assert _rel(c["y"], r["y"]) < 1e-12
    assert _rel(c["final_state"], r["final_state"]) < 1e-12


def test_chunked_without_D_and_init():
    x, dt, A, B, C, D, _ = _rand(7)
    r = exact.ssd_recurrence(x, dt, A, B, C)
    c = exact.ssd_chunked(x, dt, A, B, C, None, 8)
    assert _rel(c["y"], r["y"]) < 1e-12


def test_entering_state_is_recurrence_state_at_chunk_start():
    """P_in[c] must be the recurrent state after the last token of chunk c-1."""
    x, dt, A, B, C, D, init = _rand(9, L=16)
    c = exact.ssd_chunked(x, dt, A, B, C, D, 4, init)
    for k in range(4):
        r = exact.ssd_recurrence(x[:, :4 * k], dt[:, :4 * k], A, B, C, D, init)
        assert _rel(c["entering"][:, k], r["final_state"]) < 1e-12


def test_slab_form_matches_batched_form():
    x, dt, A, B, C, D, _ = _rand(11, L=32)
    c = exact.ssd_chunked(x, dt, A, B, C, D, 8)
    gi = exact.head_group(4, 2)
    for b in range(2):
        for h in range(4):
            s = exact.ssd_chunked_bh(x[b, :, h], dt[b, :, h], A[h], B[b, :, gi[h]],
                                     C[b, :, gi[h]], D[h], 8)
            assert _rel(s["y"], c["y"][b, :, h]) < 1e-12
            assert _rel(s["final_state"], c["final_state"][b, h]) < 1e-12


def test_reformulation_identity():
    """Eq. 7: moving the LUT from B onto X leaves the chunk state unchanged."""
    rng = np.random.default_rng(3)
    X = rng.standard_normal((16, 4))
    Bm = rng.standard_normal((16, 6))
    lut = np.exp(rng.uniform(-5, 0, 16))
    a = X.T @ (Bm * lut[:, None])
    b = (X * lut[:, None]).T @ Bm
    assert _rel(a, b) < 1e-14


def test_group_broadcast_convention():
    """Head h reads group h // (H/G); with identical groups the result is G-independent."""
    x, dt, A, B, C, D, _ = _rand(13, G=1)
    B2 = np.repeat(B, 2, axis=2)
    C2 = np.repeat(C, 2, axis=2)
    r1 = exact.ssd_recurrence(x, dt, A, B, C, D)
    r2 = exact.ssd_recurrence(x, dt, A, B2, C2, D)
    assert _rel(r1["y"], r2["y"]) < 1e-15
    assert list(exact.head_group(8, 2)) == [0, 0, 0, 0, 1, 1, 1, 1]


def test_softplus_reference_values():
    v = exact.softplus64(np.array([0.0, 1.0, -30.0, 25.0]))
    assert v[0] == np.log(2.0)
    assert abs(v[1] - np.log(1 + np.e)) < 1e-15
    assert 0 < v[2] < 1e-13
    assert v[3] == 25.0
