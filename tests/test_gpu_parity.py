"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Integer stages are compared bit for bit, each on the GPU's own inputs to that stage (stage
isolation), and end to end against the oracle's own chain; the floating-point output is held to
max|dy|/max|y| <= 1e-2 and relative L2 <= 1e-3."""
import numpy as np
import pytest

from helpers import assert_close, assert_equal, calibration, check_slab, dev, run_layer, say
from oracle import exact as oex
from oracle import int8 as oq
from paper_2608_21952_amd import synth

pytestmark = pytest.mark.gpu

ALL_TAPS = ("xs_q", "state_i32", "state_q", "decay_q", "state_in_q", "cb_i32", "cb_q",
            "scan1_i32")


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


# ---------------------------------------------------------------------------- quantize_act
@pytest.mark.parametrize("dtype", [np.float16, np.float32])
@pytest.mark.parametrize("gran", ["tensor", "group", "channel", "token"])
def test_quantize_dynamic_and_static(torch, ssdi8, dtype, gran):
    say(f"quantize_act dtype={dtype.__name__} gran={gran}")
    rng = np.random.default_rng(1)
    src = (rng.standard_normal((3, 40, 4, 128)) * np.exp(rng.uniform(-3, 3, (1, 1, 4, 1))))
    src[:, :, :, 5] *= 20
    src[1, 3] = 0
    src = src.astype(dtype)
    q_ref, a_ref = oq.quantize_act(src, gran)
    q, a = ssdi8.quantize_act(dev(src, torch), gran)
    torch.cuda.synchronize()
    assert np.array_equal(a.cpu().numpy().reshape(np.shape(a_ref)), a_ref)
    assert np.array_equal(q.cpu().numpy(), q_ref)
    q2, _ = ssdi8.quantize_act(dev(src, torch), gran, a)
    assert np.array_equal(q2.cpu().numpy(), q_ref)


@pytest.mark.parametrize("shape", [(1, 1, 4, 128), (1, 3, 64, 16), (2, 4096, 8, 128)])
@pytest.mark.parametrize("gran", ["tensor", "group", "channel"])
def test_quantize_dynamic_steps_any_block_count(torch, ssdi8, shape, gran):
    """The dynamic steps reduce per-block maxima kept in the output buffer while they fit there
    (up to one block per 4 rows, many blocks at full size) and fall back to atomic maxima when
    they do not (a single row with per-channel steps)."""
    say(f"quantize_act dynamic shape={shape} gran={gran}")
    rng = np.random.default_rng(3)
    src = rng.standard_normal(shape) * np.exp(rng.uniform(-4, 4, (1, 1, shape[2], 1)))
    src.reshape(-1)[rng.integers(0, src.size, 5)] *= 50
    src = src.astype(np.float16)
    q_ref, a_ref = oq.quantize_act(src, gran)
    q, a = ssdi8.quantize_act(dev(src, torch), gran)
    torch.cuda.synchronize()
    assert np.array_equal(a.cpu().numpy().reshape(np.shape(a_ref)), a_ref)
    assert np.array_equal(q.cpu().numpy(), q_ref)


@pytest.mark.parametrize("m", [128, 24, 7])
def test_quantize_odd_row_lengths(torch, ssdi8, m):
    say(f"quantize_act m={m}")
    rng = np.random.default_rng(2)
    src = rng.standard_normal((2, 33, 3, m)).astype(np.float16)
    alpha = np.array([0.01, 0.02, 0.5], np.float32)
    q, _ = ssdi8.quantize_act(dev(src, torch), "group", dev(alpha, torch))
    assert np.array_equal(q.cpu().numpy(), oq.quantize_act(src, "group", alpha)[0])


def test_quantize_saturates_and_empty(torch, ssdi8):
    src = np.array([[[[1000.0, -1000.0, 0.5, -0.5, 1.5, 2.5] + [0.0] * 10]]], np.float32)
    q, _ = ssdi8.quantize_act(dev(src, torch), "tensor", dev(np.ones(1, np.float32), torch))
    assert q.cpu().numpy().ravel()[:6].tolist() == [127, -127, 0, 0, 2, 2]
    e, a = ssdi8.quantize_act(torch.zeros((0, 5, 2, 16), dtype=torch.float16, device="cuda"),
                              "group")
    torch.cuda.synchronize()
    assert e.shape == (0, 5, 2, 16) and a.cpu().numpy().tolist() == [1.0, 1.0]


# ---------------------------------------------------------------------------- state_pass
@pytest.mark.parametrize("shift_round", [True, False])
@pytest.mark.parametrize("shape", [(2, 9, 3, 64, 128), (1, 1, 1, 64, 128), (3, 40, 2, 8, 4),
                                   (1, 70, 1, 64, 128)])
def test_state_pass_bitexact(torch, ssdi8, shape, shift_round):
    say(f"state_pass shape={shape} round={shift_round}")
    rng = np.random.default_rng(3)
    b, c, h, p, n = shape
    sq = rng.integers(-127, 128, shape).astype(np.int8)
    qd = rng.integers(0, 129, (b, h, c)).astype(np.int16)
    qd[:, :, ::5] = 128
    qd[:, :, 1::7] = 0
    init = rng.integers(-127, 128, (b, h, p, n)).astype(np.int8)
    scale = rng.uniform(0.01, 1.0, (h, p)).astype(np.float32)
    out = ssdi8.state_pass(dev(sq, torch), dev(qd, torch), 7, shift_round, dev(init, torch),
                           dev(scale, torch))
    torch.cuda.synchronize()
    pin_ref = np.empty_like(sq)
    fin_ref = np.empty((b, h, p, n), np.int8)
    for bi in range(b):
        for hi in range(h):
            pr, fr = oq.state_pass(sq[bi, :, hi], qd[bi, hi], init[bi, hi], 7, shift_round)
            pin_ref[bi, :, hi] = pr
            fin_ref[bi, hi] = fr
    assert np.array_equal(out["state_in_q"].cpu().numpy(), pin_ref)
    assert np.array_equal(out["final_q"].cpu().numpy(), fin_ref)
    assert np.array_equal(out["final_state"].cpu().numpy(),
                          fin_ref.astype(np.float32) * scale[None, :, :, None])


def test_state_pass_zero_chunks_copies_init(torch, ssdi8):
    rng = np.random.default_rng(4)
    init = rng.integers(-127, 128, (2, 3, 64, 128)).astype(np.int8)
    out = ssdi8.state_pass(torch.zeros((2, 0, 3, 64, 128), dtype=torch.int8, device="cuda"),
                           torch.zeros((2, 3, 0), dtype=torch.int16, device="cuda"), 7, True,
                           dev(init, torch))
    assert np.array_equal(out["final_q"].cpu().numpy(), init)


# ---------------------------------------------------------------------------- whole layer
def _check_all(g, inp, sc, cfg, **kw):
    for b in range(inp["x"].shape[0]):
        for h in range(inp["x"].shape[2]):
            check_slab(g, inp, sc, b, h, cfg.chunk, **kw)


def test_layer_tiny_all_stages(torch, ssdi8):
    cfg = synth.CONFIGS["tiny"]
    say(f"layer {cfg.name}: B={cfg.batch} L={cfg.seqlen} H={cfg.nheads} G={cfg.ngroups} fp32")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS)
    _check_all(g, inp, sc, cfg, out_dtype=np.float32)
    # whole-layer oracle (all heads at once) for the global y tolerance
    ref = oq.ssdi8_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                           sc["corr"], sc, chunk=cfg.chunk, want=("y",))
    assert_close(g["y"], ref["y"], "y (whole layer)")


@pytest.mark.parametrize("H,G", [(6, 3), (5, 1), (8, 8)])
def test_layer_ragged_fp16(torch, ssdi8, H, G):
    cfg = synth.CONFIGS["mamba2-130m"].scaled(name=f"ragged-{H}-{G}", batch=2, seqlen=768,
                                              nheads=H, ngroups=G, x_outliers=4)
    say(f"layer {cfg.name}: B=2 L=768 H={H} G={G} fp16")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS)
    _check_all(g, inp, sc, cfg)


def _small(name="variant", **kw):
    base = dict(name=name, batch=2, seqlen=512, nheads=4, ngroups=2, x_outliers=4)
    base.update(kw)
    return synth.CONFIGS["mamba2-130m"].scaled(**base)


def test_decay_skips_leave_y_unchanged(torch, ssdi8):
    """ChunkScan1 of a 32-token block whose decay factor exp(cs) is zero in fp32 is skipped
    unless its INT32 product is tapped: y must be bit-identical with and without the tap (a
    tapped call runs the separate kernels, so the single pass is held to them too).  The inputs
    decay strongly enough that both ChunkScan skips (that one, and off-diagonal blocks of the
    fp16 weights that round to zero) occur."""
    cfg = _small("decay-skip", batch=1, seqlen=1024, nheads=8, ngroups=1)
    say(f"layer {cfg.name}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    dt = np.log1p(np.exp(inp["dt_raw"].astype(np.float64)))
    cs = np.cumsum((dt * inp["A"].astype(np.float64)).reshape(1, -1, cfg.chunk, 8), axis=2)
    ends = cs[:, :, 31:-1:32]                       # cs at the last token of blocks 0..6
    assert (ends < -110).any() and (ends > -80).any()
    for path in ("separate", "single"):
        plain = run_layer(torch, ssdi8, inp, sc, path=path)
        tapped = run_layer(torch, ssdi8, inp, sc, path=path, taps=("scan1_i32",))
        assert np.array_equal(plain["y"].view(np.uint16), tapped["y"].view(np.uint16)), path
        assert np.array_equal(plain["final_state_q"], tapped["final_state_q"]), path
    ref = oq.ssdi8_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                           sc["corr"], sc, chunk=cfg.chunk, want=("y",))
    assert_close(plain["y"], ref["y"], "y (whole layer)")


def test_layer_per_head_xs_scale(torch, ssdi8):
    cfg = _small("per-head", xs_per_head=True)
    say(f"layer {cfg.name}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    assert sc["alpha_Xs"].shape == (4,)
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS)
    _check_all(g, inp, sc, cfg)


def test_layer_per_token_C(torch, ssdi8):
    cfg = _small("per-token-C")
    say(f"layer {cfg.name}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS, c_per_token=True)
    for b in range(2):
        for h in range(4):
            check_slab(g, inp, sc, b, h, 256, c_scale=g["C_scale"])


def test_layer_wide_dt_range(torch, ssdi8):
    """Raw dt over [-45, 25] on one token in eight (both sides of the [-40, 20] domain of the
    kernels' short fp64 softplus and of the threshold at 20, R17), with the domain edges
    themselves at fixed tokens: the stage outputs of the separate kernels and the single pass's
    final state match the oracle bit for bit."""
    cfg = _small("wide-dt")
    say(f"layer {cfg.name}")
    inp = synth.draw(cfg, 1)
    rng = np.random.default_rng(5)
    dt = inp["dt_raw"].copy()
    wide = rng.random(dt.shape) < 0.125
    dt[wide] = rng.uniform(-45.0, 25.0, int(wide.sum())).astype(np.float32)
    f32 = np.float32
    edges = np.array([-40.0, np.nextafter(f32(-40.0), f32(-50.0)), 20.0,
                      np.nextafter(f32(20.0), f32(30.0)), 0.0, -0.0, -45.0, 25.0], np.float32)
    dt[0, 3:3 + edges.size, 1] = edges
    dt[1, 300:300 + edges.size, 2] = edges
    inp = dict(inp, dt_raw=dt)
    sc = calibration(cfg)
    # fp32 output: with dt up to 25 a few outputs exceed the fp16 range
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS, y_dtype=torch.float32)
    for b in range(cfg.batch):
        for h in range(cfg.nheads):
            check_slab(g, inp, sc, b, h, cfg.chunk, out_dtype=np.float32)
    one = run_layer(torch, ssdi8, inp, sc, path="single", y_dtype=torch.float32,
                    taps=("state_in_q",))
    assert int(one["hand_off_timeouts"][0]) == 0
    ref = oq.ssdi8_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                           sc["corr"], sc, chunk=cfg.chunk, want=("y64", "final_q", "pin"))
    assert np.isfinite(ref["y64"]).all()
    assert_equal(one["state_in_q"], g["state_in_q"], "P_in single pass vs separate (wide dt)")
    assert_equal(one["state_in_q"], ref["pin"], "P_in single pass vs oracle (wide dt)")
    assert np.array_equal(one["final_state_q"], ref["final_q"])
    assert_equal(one["y"], g["y"], "y single pass vs separate kernels (wide dt)")
    assert_close(one["y"], ref["y64"], "y (single pass, wide dt)")


def _softplus_near_boundary(n_draw=1 << 24, rel=2.0 ** -44, seed=9):
    """Raw fp32 dt values whose fp64 softplus lies within `rel` (relative) of an fp32 rounding
    boundary: there the kernels' short softplus defers to the library's exp and log1p."""
    rng = np.random.default_rng(seed)
    x = rng.uniform(-30.0, 19.0, n_draw).astype(np.float32)
    v = oq.softplus64(x)
    m = v.astype(np.float32)
    dist = np.full(v.shape, np.inf)
    for nb in (np.nextafter(m, np.float32(np.inf)), np.nextafter(m, np.float32(-np.inf))):
        dist = np.minimum(dist, np.abs(v - (m.astype(np.float64) + nb.astype(np.float64)) / 2))
    return x[dist < rel * v]


def test_softplus_tap_bitexact(torch, ssdi8):
    """The dt the kernels use (tap dt_post) is fl32 of the fp64 softplus (R17) on every token:
    raw dt over [-45, 25], the edges of the short form's domain [-40, 20], and inputs next to an
    fp32 rounding boundary, where the short form defers to the library.  Only values that are
    ambiguous within a few fp64 ulps (the oracle's fragile rule) may differ."""
    cfg = _small("softplus-tap", batch=1, seqlen=4096, nheads=4)
    inp = synth.draw(cfg, 1)
    near = _softplus_near_boundary()
    say(f"softplus tap: {near.size} near-boundary inputs")
    assert near.size >= 4
    f32 = np.float32
    edges = np.array([-40.0, np.nextafter(f32(-40.0), f32(-50.0)), 20.0,
                      np.nextafter(f32(20.0), f32(30.0)), np.nextafter(f32(20.0), f32(0.0)),
                      0.0, -0.0, -45.0, 25.0, -1e-30, 1e-30], np.float32)
    dt = inp["dt_raw"].copy()
    flat = dt.reshape(-1)
    rng = np.random.default_rng(6)
    wide = rng.random(flat.shape) < 0.25
    flat[wide] = rng.uniform(-45.0, 25.0, int(wide.sum())).astype(np.float32)
    flat[:near.size] = near
    flat[near.size:near.size + edges.size] = edges
    inp = dict(inp, dt_raw=dt)
    sc = calibration(cfg)
    g = run_layer(torch, ssdi8, inp, sc, taps=("dt_post",), y_dtype=torch.float32)
    ref = oq.dt_post(dt, True)
    fragile = oq._ambiguous_fp32(oq.softplus64(dt)) & (dt <= 20.0)
    diff = g["dt_post"] != ref
    assert not np.any(diff & ~fragile), f"dt differs at {np.argwhere(diff & ~fragile)[:5]}"
    say(f"  {int(fragile.sum())} fragile, {int(diff.sum())} differ")
    raw = g["dt_post"].copy()
    g0 = run_layer(torch, ssdi8, inp, sc, taps=("dt_post",), dt_softplus=False,
                   y_dtype=torch.float32)
    assert np.array_equal(g0["dt_post"].view(np.uint32), dt.view(np.uint32))
    assert np.all(np.isfinite(raw))


@pytest.mark.parametrize("shift_round", [True, False])
def test_layer_floor_or_round_shift_and_init_state(torch, ssdi8, shift_round):
    cfg = _small("init", seqlen=768)
    say(f"layer {cfg.name} round={shift_round}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    init = np.random.default_rng(5).integers(-127, 128, (2, 4, 64, 128)).astype(np.int8)
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS, shift_round=shift_round, init_q=init)
    _check_all(g, inp, sc, cfg, shift_round=shift_round, init_q=init)


def test_layer_no_softplus_no_skip_no_corr_fp32_out(torch, ssdi8):
    cfg = _small("raw-dt")
    say(f"layer {cfg.name}")
    inp = synth.draw(cfg, 1)
    inp["dt_raw"] = oq.dt_post(inp["dt_raw"], True)        # pass post-softplus dt
    sc = calibration(cfg)
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS, dt_softplus=False, use_D=False,
                  use_corr=False, y_dtype=torch.float32)
    _check_all(g, inp, sc, cfg, dt_softplus=False, use_D=False, use_corr=False,
               out_dtype=np.float32)


def test_layer_saturating_scales(torch, ssdi8):
    """Step sizes far too small: every int8 stage saturates; the clamps must match exactly."""
    cfg = _small("saturate")
    say(f"layer {cfg.name}")
    inp = synth.draw(cfg, 1)
    sc = dict(calibration(cfg))
    for k, f in (("alpha_Xs", 2000), ("alpha_S", 20000), ("alpha_CB", 1000)):
        sc[k] = (np.asarray(sc[k]) / f).astype(np.float32)
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS)
    for name, least in (("xs_q", 0.05), ("state_q", 0.3), ("state_in_q", 0.1), ("cb_q", 0.3)):
        frac = float(np.mean(np.abs(g[name]) == 127))
        say(f"  saturated fraction of {name}: {frac:.3f}")
        assert frac > least, f"{name} saturates only {frac:.3f}"
    for b in range(2):
        for h in range(4):
            check_slab(g, inp, sc, b, h, 256, check_end_to_end=False)


# ---------------------------------------------------------------------------- exact cases
@pytest.mark.parametrize("A_val", [0.0, -1000.0])
def test_exact_special_cases_on_gpu(torch, ssdi8, A_val):
    """Integer-valued inputs with unit steps: the int8 path reproduces the fp64 SSD exactly."""
    say(f"special case A={A_val}")
    rng = np.random.default_rng(6)
    Bt, L, H, P, G, N = 1, 512, 2, 64, 1, 128
    dens = 0.02 if A_val == 0 else 0.3

    def tern(shape, d):
        return (rng.integers(-1, 2, shape) * (rng.random(shape) < d)).astype(np.float16)
    inp = {"x": tern((Bt, L, H, P), dens), "B": tern((Bt, L, G, N), dens),
           "C": tern((Bt, L, G, N), 0.2), "dt_raw": np.ones((Bt, L, H), np.float32),
           "A": np.full(H, A_val, np.float32), "D": np.ones(H, np.float32)}
    one = lambda *s: np.ones(s, np.float32)
    sc = {"alpha_B": one(G), "alpha_C": one(G), "alpha_Xs": one(H, P), "alpha_S": one(H, P),
          "alpha_CB": one(G), "corr": np.zeros((H, P), np.float32)}
    ref = oex.ssd_chunked(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"], 256)
    assert np.abs(ref["states"]).max() <= 127 and np.abs(ref["entering"]).max() <= 127
    assert np.abs(ref["final_state"]).max() <= 127 and np.abs(ref["y"]).max() < 2048
    g = run_layer(torch, ssdi8, inp, sc, taps=ALL_TAPS, dt_softplus=False, y_dtype=torch.float32)
    assert np.array_equal(g["y"].astype(np.float64), ref["y"])
    assert np.array_equal(g["final_state_q"].astype(np.float64), ref["final_state"])


# ---------------------------------------------------------------------------- ABI behaviour
def test_determinism_and_resume(torch, ssdi8):
    cfg = _small("resume", seqlen=1024)
    say(f"determinism/resume {cfg.name}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    a = run_layer(torch, ssdi8, inp, sc, taps=("state_in_q",))
    b = run_layer(torch, ssdi8, inp, sc, taps=("state_in_q",))
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    half = {k: (v[:, :512] if k in ("x", "dt_raw", "B", "C") else v) for k, v in inp.items()}
    rest = {k: (v[:, 512:] if k in ("x", "dt_raw", "B", "C") else v) for k, v in inp.items()}
    # resuming from the int8 final state gives the same results, on both paths (the single pass
    # and the separate kernels; their y differ only by the rounding of the output tables)
    for path in ("separate", "single"):
        whole = run_layer(torch, ssdi8, inp, sc, path=path)
        h1 = run_layer(torch, ssdi8, half, sc, path=path)
        h2 = run_layer(torch, ssdi8, rest, sc, init_q=h1["final_state_q"], path=path)
        assert np.array_equal(np.concatenate([h1["y"], h2["y"]], axis=1), whole["y"])
        assert np.array_equal(h2["final_state_q"], a["final_state_q"])
        assert np.array_equal(whole["final_state_q"], a["final_state_q"])


def test_empty_sequence_returns_initial_state(torch, ssdi8):
    rng = np.random.default_rng(7)
    H, P, N, G = 4, 64, 128, 1
    init = rng.integers(-127, 128, (2, H, P, N)).astype(np.int8)
    aS = rng.uniform(0.1, 1, (H, P)).astype(np.float32)
    z = lambda *s, dt=torch.float16: torch.zeros(s, dtype=dt, device="cuda")
    out = ssdi8.ssd_chunk_scan(
        z(2, 0, H, P), z(2, 0, H, dt=torch.float32), dev(np.full(H, -1, np.float32), torch),
        z(2, 0, G, N, dt=torch.int8), z(2, 0, G, N, dt=torch.int8), dev(np.ones(G, np.float32), torch),
        dev(np.ones(G, np.float32), torch), dev(np.ones((H, P), np.float32), torch),
        dev(aS, torch), dev(np.ones(G, np.float32), torch), init_state_q=dev(init, torch))
    torch.cuda.synchronize()
    assert np.array_equal(out["final_state_q"].cpu().numpy(), init)
    assert np.array_equal(out["final_state"].cpu().numpy(),
                          init.astype(np.float32) * aS[None, :, :, None])


def test_invalid_arguments_raise(torch, ssdi8):
    cfg = _small("bad")
    inp = synth.draw(cfg, 1)
    x = dev(inp["x"], torch)
    f = lambda *s: torch.ones(s, dtype=torch.float32, device="cuda")
    q = torch.zeros((2, 512, 2, 128), dtype=torch.int8, device="cuda")
    with pytest.raises(ssdi8.SSDi8Error) as e:     # seqlen not a multiple of the chunk
        ssdi8.ssd_chunk_scan(x[:, :300].contiguous(), f(2, 300, 4), f(4), q[:, :300].contiguous(),
                             q[:, :300].contiguous(), f(2), f(2), f(4, 64), f(4, 64), f(2))
    assert e.value.status == ssdi8.ERR_SHAPE
    with pytest.raises(ssdi8.SSDi8Error) as e:     # unsupported head dim
        ssdi8.ssd_chunk_scan(x[..., :32].contiguous(), f(2, 512, 4), f(4), q, q, f(2), f(2),
                             f(4, 32), f(4, 32), f(2))
    assert e.value.status == ssdi8.ERR_UNSUPPORTED
    with pytest.raises(ssdi8.SSDi8Error) as e:
        ssdi8.ssd_chunk_scan(x, f(2, 512, 4), f(4), q, q, f(2), f(2), f(4, 64), f(4, 64), f(2),
                             decay_shift=0)
    assert e.value.status == ssdi8.ERR_ARG


def test_graph_replay_matches_eager(torch, ssdi8):
    """One layer captured as a HIP graph: every replay (with eager work and synchronisations in
    between) reproduces the eager outputs bit for bit."""
    cfg = _small("graph", seqlen=768)
    say(f"graph replay {cfg.name}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    eager = run_layer(torch, ssdi8, inp, sc, taps=("state_in_q", "cb_q"))
    x, dt = dev(inp["x"], torch), dev(inp["dt_raw"], torch)
    Bf, Cf = dev(inp["B"], torch), dev(inp["C"], torch)
    layer = ssdi8.SSDi8Layer(inp["A"], inp["D"], sc["corr"], sc, device="cuda")
    y = torch.empty_like(x)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layer(x, dt, Bf, Cf, y=y)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = layer(x, dt, Bf, Cf, y=y, taps=("state_in_q", "cb_q"))
    for rep in range(4):
        y.zero_()
        out["state_in_q"].zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), eager["y"]), f"replay {rep}: y differs"
        assert np.array_equal(out["state_in_q"].cpu().numpy(), eager["state_in_q"]), rep
        assert np.array_equal(out["final_state_q"].cpu().numpy(), eager["final_state_q"]), rep


def test_mfma_probe_counts_and_runs(torch, ssdi8):
    """The measurement helper: its op count is the launch's (workgroups x 4 waves x 4 chains x
    iterations x 2 M N K) and it runs to completion for both kinds."""
    import ctypes
    for kind, mnk in ((0, 32 * 32 * 32), (1, 32 * 32 * 16)):
        out = torch.zeros(8 * 256, dtype=torch.int32 if kind == 0 else torch.float32,
                          device="cuda")
        ops = ctypes.c_int64()
        st = ssdi8.lib().ssdi8_mfma_probe(kind, 100, 8, out.data_ptr(), ctypes.byref(ops), None)
        torch.cuda.synchronize()
        assert st == 0 and ops.value == 8 * 4 * 4 * 100 * 2 * mnk
    assert ssdi8.mfma_peak("int8", iters=200, blocks=256, reps=1) > 0
