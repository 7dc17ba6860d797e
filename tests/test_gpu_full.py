"""GPU parity at the full workload sizes, in the launch configuration the benchmark times.

The oracle cannot afford whole layers at these sizes, so it checks (a) sampled (batch, head)
slabs stage by stage and end to end, and (b) properties that hold at any size and are cheap
in NumPy for every head and chunk: Q(Decay), the INT8 state passing recomputed from the
GPU's own S_q, and CB_q recomputed from the GPU's own B_q, C_q."""
import os

import numpy as np
import pytest

from helpers import CALIB_DIR, assert_equal, calibration, check_slab, run_layer, say
from oracle import exact as oex
from oracle import int8 as oq
from paper_2608_21952_amd import synth

pytestmark = pytest.mark.gpu

TAPS = ("xs_q", "state_q", "decay_q", "state_in_q", "cb_q")


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


def _sample_heads(cfg):
    H, B = cfg.nheads, cfg.batch
    picks = {(0, 0), (B - 1, H - 1), (B // 2, H // 2 + 1), (0, H // cfg.ngroups)}
    return sorted((b, h % H) for b, h in picks)


@pytest.mark.parametrize("name", ["mamba2-130m", "mamba2-2.7b", "mamba2-8b-g8", "long-64k"])
def test_full_size_layer(torch, ssdi8, name):
    cfg = synth.CONFIGS[name]
    assert os.path.exists(os.path.join(CALIB_DIR, name + ".npz")), "stored calibration missing"
    say(f"full-size layer {name}: B={cfg.batch} L={cfg.seqlen} H={cfg.nheads} G={cfg.ngroups}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    g = run_layer(torch, ssdi8, inp, sc, taps=TAPS)
    Q, k = cfg.chunk, 7
    B, L, H, P = inp["x"].shape
    G, N = inp["B"].shape[2], inp["B"].shape[3]
    nc = L // Q
    gi = oex.head_group(H, G)
    # (b) whole-tensor properties
    dt32 = oq.dt_post(inp["dt_raw"], True)                              # (B,L,H)
    dA = (dt32 * np.asarray(inp["A"], np.float32)[None, None, :]).reshape(B, nc, Q, H)
    cs_last = np.moveaxis(oq.exact_prefix_sum64(np.moveaxis(dA, 2, 3))[..., -1], 1, 2)
    qd = np.rint(np.exp(cs_last) * 2.0 ** k).astype(np.int32)           # (B,H,c)
    bad = np.argwhere(g["decay_q"] != qd)
    for (b, h, c) in bad:     # only values at an fp rounding boundary may differ (none expected)
        frag = oq.fragile_tokens(inp["dt_raw"][b, :, h], inp["A"][h], Q, True, k)
        assert frag[c * Q:(c + 1) * Q].any(), f"Q(Decay) differs at b={b} h={h} c={c}"
    if len(bad):
        say(f"  Q(Decay): {len(bad)} fragile chunks differ")
    say("  Q(Decay) all heads: ok")
    pin, fin = oq.state_pass(np.moveaxis(g["state_q"], 1, 0),
                             np.moveaxis(g["decay_q"], 2, 0), None, k)
    assert_equal(g["state_in_q"], np.moveaxis(pin, 0, 1), "P_in, all heads")
    assert_equal(g["final_state_q"], fin, "final int8 state, all heads")
    say("  StatePassing all heads: ok")
    for b in range(B):
        for gg in range(G):
            cb = oq.chunk_bmm(g["Cq"][b, :, gg], g["Bq"][b, :, gg], sc["alpha_C"][gg],
                              sc["alpha_B"][gg], sc["alpha_CB"][gg], Q)
            assert_equal(g["cb_q"][b, :, gg], cb["CBq"], f"CB_q b={b} g={gg}")
    say("  CB_q all chunks: ok")
    # (a) sampled slabs, stage by stage and end to end
    for (b, h) in _sample_heads(cfg):
        say(f"  slab b={b} h={h} (group {gi[h]})")
        check_slab(g, inp, sc, b, h, Q)
