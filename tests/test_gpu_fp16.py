"""GPU parity of the FP16 baseline (ssdi8_ssd_chunk_scan_fp16) against its oracle
(oracle/fp16.py, itself pinned against the fp64 forms): y within the stated tolerance and the
fp32 final state within 1e-5 relative L2, whole layers and sampled full-size slabs."""
import dataclasses

import numpy as np
import pytest

from helpers import assert_close, dev, rel_errors, say
from oracle import fp16 as ofp
from paper_2608_21952_amd import synth

pytestmark = pytest.mark.gpu

STATE_RELL2 = 1e-5


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


def _run(torch, ssdi8, inp, init=None, y_dtype=None):
    f = lambda v: dev(np.asarray(v, np.float32), torch)
    return ssdi8.ssd_chunk_scan_fp16(dev(inp["x"], torch), f(inp["dt_raw"]), f(inp["A"]),
                                     dev(inp["B"], torch), dev(inp["C"], torch), D=f(inp["D"]),
                                     init_state=None if init is None else f(init),
                                     y_dtype=y_dtype)


def _check_state(gpu, ref, what):
    _, rel = rel_errors(gpu, ref)
    say(f"  {what}: relL2 = {rel:.3e}")
    assert rel <= STATE_RELL2, f"{what}: relative L2 {rel:.3e} > {STATE_RELL2}"


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("mamba2-130m", dict(batch=2, seqlen=1024, nheads=8)),
    ("mamba2-8b-g8", dict(batch=1, seqlen=768, nheads=16, ngroups=4)),
])
def test_fp16_layer_matches_oracle(torch, ssdi8, name, over):
    cfg = dataclasses.replace(synth.CONFIGS[name], name=name + "-fp16", **over)
    say(f"fp16 layer {cfg.name}: B={cfg.batch} L={cfg.seqlen} H={cfg.nheads} G={cfg.ngroups} "
        f"{cfg.dtype}")
    inp = synth.draw(cfg, 1)
    g = _run(torch, ssdi8, inp)
    ref = ofp.ssd_fp16_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                               chunk=cfg.chunk)
    assert_close(g["y"].float().cpu().numpy(), ref["y64"], "y")
    _check_state(g["final_state"].cpu().numpy(), ref["final_state"], "final state")


def test_fp16_initial_state_and_fp32_output(torch, ssdi8):
    cfg = dataclasses.replace(synth.CONFIGS["mamba2-130m"], name="fp16-init", batch=2,
                              seqlen=512, nheads=4)
    inp = synth.draw(cfg, 2)
    rng = np.random.default_rng(4)
    init = rng.standard_normal((2, 4, 64, 128)).astype(np.float32)
    g = _run(torch, ssdi8, inp, init=init, y_dtype=torch.float32)
    ref = ofp.ssd_fp16_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                               chunk=cfg.chunk, init=init)
    assert g["y"].dtype == torch.float32
    assert_close(g["y"].cpu().numpy(), ref["y64"], "y (fp32 out, initial state)")
    _check_state(g["final_state"].cpu().numpy(), ref["final_state"], "final state")


@pytest.mark.parametrize("name", ["mamba2-130m", "mamba2-2.7b"])
def test_fp16_full_size_sampled_slabs(torch, ssdi8, name):
    """Full-size layers, the 2.7B-shaped one with x and y streamed through the caches."""
    cfg = synth.CONFIGS[name]
    say(f"fp16 layer full size {name}")
    inp = synth.draw(cfg, 1)
    g = _run(torch, ssdi8, inp)
    y = g["y"].float().cpu().numpy()
    fin = g["final_state"].cpu().numpy()
    picks = [(0, 0), (cfg.batch - 1, cfg.nheads - 1), (cfg.batch // 2, cfg.nheads // 2)]
    ref = ofp.ssd_fp16_forward(inp["x"], inp["dt_raw"], inp["A"], inp["B"], inp["C"], inp["D"],
                               chunk=cfg.chunk, heads=picks)
    for (b, h) in picks:
        r = ref["slabs"][(b, h)]
        assert_close(y[b, :, h], r["y64"], f"y slab ({b},{h})")
        _check_state(fin[b, h], r["final"], f"final state slab ({b},{h})")


def test_fp16_empty_sequence_returns_initial_state(torch, ssdi8):
    init = torch.randn((2, 4, 64, 128), device="cuda")
    z = lambda *s: torch.zeros(s, dtype=torch.float32, device="cuda")
    h16 = lambda *s: torch.zeros(s, dtype=torch.float16, device="cuda")
    out = ssdi8.ssd_chunk_scan_fp16(h16(2, 0, 4, 64), z(2, 0, 4), z(4), h16(2, 0, 1, 128),
                                    h16(2, 0, 1, 128), init_state=init)
    assert torch.equal(out["final_state"], init)
