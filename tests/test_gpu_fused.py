"""The single-pass kernel (ChunkState, StatePassing and ChunkScan in one launch; each chunk
obtains the int8 state entering it from the chunks before it in its sequence through memory and
a flag per chunk).

Bar: every entering state P_in[c] of every chunk (the state_in_q tap, which the single pass
fills from its workspace without switching paths) and the final int8 state bit-identical to
the oracle's StatePassing (Eq. 9) run on the separate kernels' chunk-local S_q and Q(Decay)
(themselves checked stage by stage against the oracle in the full-size parity tests), and to the
oracle's end-to-end chain on the small cases; y bit-identical to the separate kernels (both
compute dt, the ChunkScan tables and the products in the same order) and within the y tolerance
of the oracle; no wait runs out (both the device counter of the call and the one in the
workspace); repeated calls on one workspace and graph replays reproduce the results exactly."""
import numpy as np
import pytest

from helpers import assert_close, assert_equal, calibration, dev, run_layer, say
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


def _workspace(torch, ssdi8, cfg):
    d = ssdi8.dims(cfg.batch, cfg.seqlen, cfg.nheads, cfg.ngroups)
    return torch.empty(ssdi8.workspace_size(d), dtype=torch.uint8, device="cuda")


# hand-off words: a ticket counter per 128-byte line for up to 64 sequence classes, the count of
# waits that ran out on the next line, then the flags
SYNC_LINE, SYNC_CLASSES = 32, 64
SYNC_WAIT = SYNC_CLASSES * SYNC_LINE
SYNC_FLAGS = SYNC_WAIT + SYNC_LINE


def _timed_out_waits(ws, cfg):
    """The hand-off words are the last region of the workspace, padded to 256 bytes."""
    nc = cfg.seqlen // cfg.chunk
    n = SYNC_FLAGS + cfg.batch * cfg.nheads * nc
    off = ws.numel() - ((4 * n + 255) // 256) * 256
    words = ws[off:off + 4 * (SYNC_WAIT + 1)].cpu().numpy().view(np.int32)
    return int(words[SYNC_WAIT])


def _no_timeouts(out, ws=None, cfg=None):
    assert int(out["hand_off_timeouts"][0]) == 0, "a hand-off wait ran out (device counter)"
    if ws is not None:
        assert _timed_out_waits(ws, cfg) == 0, "a hand-off wait ran out (workspace counter)"


def _check_pin_against_separate(one, sep, init=None, k=7, shift_round=True):
    """The single pass's entering states equal the separate kernels' and the oracle's Eq. 9
    chain over the separate kernels' chunk-local S_q and Q(Decay), for every (b, h)."""
    assert_equal(one["state_in_q"], sep["state_in_q"], "P_in single pass vs separate kernels")
    Bt, _, H = one["state_in_q"].shape[:3]
    for b in range(Bt):
        for h in range(H):
            i0 = None if init is None else init[b, h]
            pin, fin = oq.state_pass(sep["state_q"][b, :, h], sep["decay_q"][b, h], i0, k,
                                     shift_round)
            assert_equal(one["state_in_q"][b, :, h], pin, f"P_in[b={b},h={h}] vs oracle Eq. 9")
            assert_equal(one["final_state_q"][b, h], fin, f"final_q[b={b},h={h}] vs oracle")


SEP_TAPS = ("state_q", "decay_q", "state_in_q")


def _small(name, **kw):
    base = dict(name=name, batch=2, seqlen=1024, nheads=8, ngroups=2, x_outliers=4)
    base.update(kw)
    return synth.CONFIGS["mamba2-130m"].scaled(**base)


CASES = [
    _small("fused-130m-like", ngroups=1),
    _small("fused-groups", nheads=6, ngroups=3, seqlen=1536),
    _small("fused-per-head", xs_per_head=True, seqlen=768),
    _small("fused-one-chunk", seqlen=256, batch=3),
    # slowly decaying heads (A in [-0.14, -0.018]): Q(Decay) > 0 on every chunk, so every
    # entering state comes through the look-back hand-off
    _small("fused-slow-decay", seqlen=2048, a_lo=-4.0, a_hi=-2.0),
    # the 64K-token layer's mix (A in [-16, -0.018]): early zero-decay publications and
    # look-back chains side by side
    _small("fused-mixed-decay", seqlen=2048, nheads=16, a_lo=-4.0),
]


@pytest.mark.parametrize("cfg", CASES, ids=lambda c: c.name)
def test_single_pass_matches_separate_kernels_and_oracle(torch, ssdi8, cfg):
    say(f"single pass {cfg.name}: B={cfg.batch} L={cfg.seqlen} H={cfg.nheads} G={cfg.ngroups}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    ws = _workspace(torch, ssdi8, cfg)
    f32 = torch.float32
    one = run_layer(torch, ssdi8, inp, sc, y_dtype=f32, workspace=ws, path="single",
                    taps=("state_in_q",))
    _no_timeouts(one, ws, cfg)
    sep = run_layer(torch, ssdi8, inp, sc, y_dtype=f32, path="separate", taps=SEP_TAPS)
    _no_timeouts(sep)
    _check_pin_against_separate(one, sep)
    assert np.array_equal(one["final_state"], sep["final_state"])
    assert_equal(one["y"], sep["y"], "y single pass vs separate kernels")
    ref = oq.ssdi8_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                           sc["corr"], sc, chunk=cfg.chunk, want=("y64", "final_q", "pin"))
    assert_equal(one["state_in_q"], ref["pin"], "P_in single pass vs oracle chain")
    assert_equal(one["final_state_q"], ref["final_q"], "final_q vs oracle chain")
    assert_close(one["y"], ref["y64"], "y (single pass, fp32 out)")
    # the fp16 output of the single pass as well
    hq = run_layer(torch, ssdi8, inp, sc, workspace=ws, path="single", taps=("state_in_q",))
    _no_timeouts(hq, ws, cfg)
    assert_close(hq["y"], ref["y64"], "y (single pass, fp16 out)")
    assert_equal(hq["state_in_q"], ref["pin"], "P_in (fp16 output run)")
    assert np.array_equal(hq["final_state_q"], ref["final_q"])


@pytest.mark.parametrize("shift_round,shift", [(False, 7), (True, 6), (True, 8), (False, 11)])
def test_single_pass_variants(torch, ssdi8, shift_round, shift):
    """Initial state, floor or rounded shift of another width, per-token C steps, raw dt, no skip,
    no correction."""
    cfg = _small("fused-variants", seqlen=768, nheads=4)
    say(f"single pass variants round={shift_round} k={shift}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    init = np.random.default_rng(11).integers(-127, 128, (2, 4, 64, 128)).astype(np.int8)
    kw = dict(shift_round=shift_round, decay_shift=shift, init_q=init, c_per_token=True,
              y_dtype=torch.float32)
    one = run_layer(torch, ssdi8, inp, sc, path="single", taps=("state_in_q",), **kw)
    _no_timeouts(one)
    sep = run_layer(torch, ssdi8, inp, sc, path="separate", taps=SEP_TAPS, **kw)
    _check_pin_against_separate(one, sep, init, shift, shift_round)
    assert_equal(one["y"], sep["y"], "y single pass vs separate kernels")
    raw = dict(inp)
    raw["dt_raw"] = oq.dt_post(inp["dt_raw"], True)
    kw2 = dict(dt_softplus=False, use_D=False, use_corr=False, init_q=init,
               shift_round=shift_round, decay_shift=shift, y_dtype=torch.float32)
    one = run_layer(torch, ssdi8, raw, sc, path="single", taps=("state_in_q",), **kw2)
    _no_timeouts(one)
    ref = oq.ssdi8_forward(raw["x"], raw["dt_raw"], raw["A"], raw["B"], raw["C"],
                           np.zeros(4, np.float32), np.zeros((4, 64), np.float32), sc,
                           chunk=cfg.chunk, dt_softplus=False, k=shift, shift_round=shift_round,
                           init_q=init, want=("y64", "final_q", "pin"))
    assert_equal(one["state_in_q"], ref["pin"], "P_in vs oracle chain (raw dt, init state)")
    assert np.array_equal(one["final_state_q"], ref["final_q"])
    assert_close(one["y"], ref["y64"], "y (raw dt, no skip, no correction)")


def test_single_pass_repeats_and_graph_replays(torch, ssdi8):
    cfg = _small("fused-graph", seqlen=1280)
    say(f"single pass repeats / graph {cfg.name}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    ws = _workspace(torch, ssdi8, cfg)
    first = run_layer(torch, ssdi8, inp, sc, workspace=ws, path="single", taps=("state_in_q",))
    for rep in range(3):
        again = run_layer(torch, ssdi8, inp, sc, workspace=ws, path="single",
                          taps=("state_in_q",))
        _no_timeouts(again, ws, cfg)
        for k in ("y", "final_state_q", "final_state", "state_in_q"):
            assert np.array_equal(again[k], first[k]), (rep, k)
    x, dt = dev(inp["x"], torch), dev(inp["dt_raw"], torch)
    Bf, Cf = dev(inp["B"], torch), dev(inp["C"], torch)
    layer = ssdi8.SSDi8Layer(inp["A"], inp["D"], sc["corr"], sc, device="cuda")
    y = torch.empty_like(x)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layer(x, dt, Bf, Cf, y=y, path="single")      # eager: checks the hand-off counter
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = layer(x, dt, Bf, Cf, y=y, path="single")
    for rep in range(4):
        y.zero_()
        out["final_state_q"].zero_()
        layer.timeouts.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), first["y"]), f"replay {rep}: y differs"
        assert np.array_equal(out["final_state_q"].cpu().numpy(), first["final_state_q"]), rep
        assert layer.hand_off_timeouts() == 0, f"replay {rep}: counter not cleared or a wait ran out"



@pytest.mark.parametrize("name", ["mamba2-130m", "mamba2-2.7b", "mamba2-8b-g8", "long-64k"])
def test_single_pass_full_size_replays_are_identical(torch, ssdi8, name):
    """At the benchmark sizes, in the launch configuration the benchmark times (one captured
    graph of ChunkBMM and the single pass, replayed back to back): every replay reproduces the
    eager call's y and final int8 state bit for bit, and no wait runs out."""
    cfg = synth.CONFIGS[name]
    reps = 30
    say(f"single pass full size {name}: {reps} graph replays against the eager call")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    x, dt = dev(inp["x"], torch), dev(inp["dt_raw"], torch)
    Bf, Cf = dev(inp["B"], torch), dev(inp["C"], torch)
    layer = ssdi8.SSDi8Layer(inp["A"], inp["D"], sc["corr"], sc, device="cuda")
    y = torch.empty_like(x)
    first = layer(x, dt, Bf, Cf, y=y)
    torch.cuda.synchronize()
    assert layer.hand_off_timeouts() == 0
    y_ref, fq_ref = y.clone(), first["final_state_q"].clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        layer(x, dt, Bf, Cf, y=y)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = layer(x, dt, Bf, Cf, y=y)
    for rep in range(reps):
        y.zero_()
        out["final_state_q"].zero_()
        layer.timeouts.fill_(-1)
        g.replay()
        torch.cuda.synchronize()
        assert layer.hand_off_timeouts() == 0, f"replay {rep}: a wait ran out"
        assert torch.equal(y, y_ref), f"replay {rep}: y differs from the eager call"
        assert torch.equal(out["final_state_q"], fq_ref), f"replay {rep}: final_q differs"
    del y, y_ref, x

def _fp16_overflow_matches_oracle(y16, y64, what):
    """Where the oracle's fp64 output rounds beyond the fp16 range (|y| >= 65520) the fp16
    output must be the infinity of the same sign, and finite elsewhere, except within the
    output tolerance of that rounding boundary; returns the mask of agreed infinities."""
    g_inf = ~np.isfinite(y16.astype(np.float32))
    r16 = y64.astype(np.float16)
    r_inf = ~np.isfinite(r16.astype(np.float32))
    near = np.abs(np.abs(y64) - 65520.0) <= 1e-3 * np.abs(y64).max()
    bad = (g_inf != r_inf) & ~near
    assert not bad.any(), f"{what}: {int(bad.sum())} fp16 overflow positions differ from the oracle"
    both = g_inf & r_inf
    assert np.array_equal(np.sign(y16[both].astype(np.float32)), np.sign(y64[both])), what
    if both.any():
        say(f"  {what}: {int(both.sum())} outputs beyond the fp16 range, as in the oracle")
    return g_inf | r_inf


@pytest.mark.parametrize("name", ["mamba2-130m", "mamba2-2.7b", "mamba2-8b-g8", "long-64k"])
def test_single_pass_full_size(torch, ssdi8, name):
    """At the benchmark sizes: every entering state and the final int8 state bit-identical to the
    oracle's Eq. 9 chain over the separate kernels' S_q and Q(Decay); y bit-identical to the
    separate kernels; y within the y tolerance of the oracle on sampled slabs, in fp16 (the
    output the benchmark writes; outputs beyond the fp16 range compared with the oracle's own
    fp16 rounding) and in fp32 (no overflow, nothing masked); no wait ran out."""
    cfg = synth.CONFIGS[name]
    say(f"single pass full size {name}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    ws = _workspace(torch, ssdi8, cfg)
    one = run_layer(torch, ssdi8, inp, sc, workspace=ws, path="single", taps=("state_in_q",))
    _no_timeouts(one, ws, cfg)
    sep = run_layer(torch, ssdi8, inp, sc, path="separate", taps=SEP_TAPS)
    _check_pin_against_separate(one, sep)
    assert_equal(one["y"], sep["y"], "y single pass vs separate kernels (fp16)")
    del sep
    picks = [(0, 0), (cfg.batch - 1, cfg.nheads - 1), (cfg.batch // 2, cfg.nheads // 2)]
    ref = oq.ssdi8_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                           sc["corr"], sc, chunk=cfg.chunk, heads=picks, want=("y64",))
    for (b, h) in picks:
        y16, y64 = one["y"][b, :, h], ref["slabs"][(b, h)]["y64"]
        inf = _fp16_overflow_matches_oracle(y16, y64, f"y slab ({b},{h})")
        assert_close(np.where(inf, 0, y16), np.where(inf, 0, y64), f"y slab ({b},{h}) fp16")
    del one
    f = run_layer(torch, ssdi8, inp, sc, workspace=ws, path="single", y_dtype=torch.float32)
    _no_timeouts(f, ws, cfg)
    for (b, h) in picks:
        assert_close(f["y"][b, :, h], ref["slabs"][(b, h)]["y64"], f"y slab ({b},{h}) fp32")


@pytest.mark.parametrize("batch,nheads,ngroups,nchunks", [(1, 1, 1, 16), (1, 3, 1, 5), (3, 3, 3, 3),
                                                          (1, 9, 3, 6)])
def test_single_pass_few_sequences(torch, ssdi8, batch, nheads, ngroups, nchunks):
    """Fewer sequences than ticket classes (most classes empty, their workgroups draw items from
    the others) and class sizes that differ by one: every chain still completes, no wait runs
    out, and the results equal the separate kernels' and the oracle's."""
    cfg = _small(f"few-{batch}x{nheads}", batch=batch, nheads=nheads, ngroups=ngroups,
                 seqlen=256 * nchunks, x_outliers=1)
    say(f"single pass few sequences: B={batch} H={nheads} G={ngroups} chunks={nchunks}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    ws = _workspace(torch, ssdi8, cfg)
    one = run_layer(torch, ssdi8, inp, sc, y_dtype=torch.float32, workspace=ws, path="single",
                    taps=("state_in_q",))
    _no_timeouts(one, ws, cfg)
    sep = run_layer(torch, ssdi8, inp, sc, y_dtype=torch.float32, path="separate", taps=SEP_TAPS)
    _check_pin_against_separate(one, sep)
    assert_equal(one["y"], sep["y"], "y single pass vs separate kernels")
    ref = oq.ssdi8_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                           sc["corr"], sc, chunk=cfg.chunk, want=("y64", "final_q", "pin"))
    assert_equal(one["state_in_q"], ref["pin"], "P_in vs oracle chain")
    assert np.array_equal(one["final_state_q"], ref["final_q"])
    assert_close(one["y"], ref["y64"], "y (few sequences)")
