"""Per-module timing of ssdi8_ssd_chunk_scan (its stage_events argument): passing the events
changes no result on either path, and every event comes back recorded, in stream order, with
ChunkBMM's and the ChunkScan kernel's own intervals (set by their dispatch) non-empty."""
import numpy as np
import pytest

from helpers import assert_equal, calibration, dev, say
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


@pytest.mark.parametrize("path", ["single", "separate"])
def test_stage_events_change_nothing_and_come_in_order(torch, ssdi8, path):
    cfg = synth.CONFIGS["mamba2-130m"].scaled(name="stage-events", batch=2, seqlen=1024,
                                              nheads=8, ngroups=2)
    say(f"stage events, path {path}: B={cfg.batch} L={cfg.seqlen} H={cfg.nheads}")
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    f32 = lambda v: dev(np.asarray(v, np.float32), torch)
    x, dt, B, C = (dev(inp[k], torch) for k in ("x", "dt_raw", "B", "C"))
    scales = [f32(sc[k]) for k in ("alpha_B", "alpha_C", "alpha_Xs", "alpha_S", "alpha_CB")]

    def call(events=None):
        out = ssdi8.ssd_chunk_scan(x, dt, f32(inp["A"]), None, None, *scales, D=f32(inp["D"]),
                                   corr=f32(sc["corr"]), B=B, C=C, path=path,
                                   stage_events=events)
        torch.cuda.synchronize()
        return {k: v.cpu().numpy() for k, v in out.items()}

    ref = call()
    ev = ssdi8.HipEvents(5)
    try:
        out = call(ev.group(0))
        for k in ("y", "final_state_q", "final_state"):
            assert_equal(out[k], ref[k], f"{k} with stage events vs without")
        since = [ev.elapsed_ms(0, i) for i in range(5)]   # raises if one was not recorded
        assert since[0] == 0.0
        assert all(b >= a for a, b in zip(since, since[1:])), since
        assert ev.elapsed_ms(0, 1) > 0.0, "ChunkBMM's interval is empty"
        assert ev.elapsed_ms(3, 4) > 0.0, "the ChunkScan kernel's interval is empty"
    finally:
        ev.close()
