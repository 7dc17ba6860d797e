"""ssdi8_ssd_chunk_scan_noalloc: the SSD layer with the library's static per-GPU scratch instead of
a caller workspace, for callers that cannot allocate.  Its results must equal those of
ssdi8_ssd_chunk_scan with a workspace, bit for bit (the same kernels on the same inputs): y, the
final int8 and fp32 states and the entering-state tap, on both kernel paths, for two calls in a
row whose second one is smaller (the scratch keeps the first call's contents, so everything the
second call reads must be its own), and after a larger call on a workspace; sizes beyond the
scratch are refused before anything runs."""
import numpy as np
import pytest

from helpers import calibration, dev, say
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


def _layer_inputs(torch, cfg):
    inp = synth.draw(cfg, 1)
    sc = calibration(cfg)
    f32 = lambda a: dev(np.asarray(a, np.float32), torch)
    args = (dev(inp["x"], torch), dev(inp["dt_raw"], torch), f32(inp["A"]), None, None,
            f32(sc["alpha_B"]), f32(sc["alpha_C"]), f32(sc["alpha_Xs"]), f32(sc["alpha_S"]),
            f32(sc["alpha_CB"]))
    kw = dict(D=f32(inp["D"]), corr=f32(sc["corr"]), B=dev(inp["B"], torch),
              C=dev(inp["C"], torch), taps=("state_in_q",))
    return args, kw


def _run(torch, fn, args, kw, path):
    to = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    out = fn(*args, path=path, hand_off_timeouts=to, **kw)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    assert int(res["hand_off_timeouts"][0]) == 0
    return res


def _same(a, b, what):
    for k in ("y", "final_state_q", "final_state", "state_in_q"):
        assert np.array_equal(a[k], b[k]), f"{what}: {k} differs"


CFGS = [
    synth.CONFIGS["mamba2-130m"].scaled(name="noalloc-first", batch=2, seqlen=2048, nheads=16,
                                        ngroups=2, x_outliers=8),
    synth.CONFIGS["mamba2-130m"].scaled(name="noalloc-second", batch=1, seqlen=768, nheads=6,
                                        ngroups=3, x_outliers=3),
]


@pytest.mark.parametrize("path", ["single", "separate"])
def test_noalloc_equals_workspace_entry_point_two_calls(torch, ssdi8, path):
    """Two calls in a row through the no-allocation entry point, the second smaller, each equal
    to the workspace entry point on the same inputs."""
    for cfg in CFGS:
        say(f"noalloc {path} {cfg.name}: B={cfg.batch} L={cfg.seqlen} H={cfg.nheads} "
            f"G={cfg.ngroups}")
        args, kw = _layer_inputs(torch, cfg)
        got = _run(torch, ssdi8.ssd_chunk_scan_noalloc, args, kw, path)
        ref = _run(torch, ssdi8.ssd_chunk_scan, args, kw, path)
        _same(got, ref, f"{cfg.name} ({path})")


def test_noalloc_after_a_larger_workspace_call_and_in_a_graph(torch, ssdi8):
    """A graph captured around the no-allocation call (its first call on the device happened
    outside the capture) replays to the same results as eager calls."""
    cfg = CFGS[1]
    args, kw = _layer_inputs(torch, cfg)
    ref = _run(torch, ssdi8.ssd_chunk_scan, args, kw, "auto")
    eager = _run(torch, ssdi8.ssd_chunk_scan_noalloc, args, kw, "auto")
    _same(eager, ref, "eager")
    x = args[0]
    y = torch.empty_like(x)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    kw2 = dict(kw)
    kw2.pop("taps")
    with torch.cuda.stream(side):
        ssdi8.ssd_chunk_scan_noalloc(*args, y=y, **kw2)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = ssdi8.ssd_chunk_scan_noalloc(*args, y=y, **kw2)
    for rep in range(3):
        y.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), ref["y"]), f"replay {rep}: y differs"
        assert np.array_equal(out["final_state_q"].cpu().numpy(), ref["final_state_q"]), rep


def test_noalloc_refuses_sizes_beyond_its_scratch(ssdi8):
    cfg = synth.CONFIGS["long-64k"]
    d = ssdi8.dims(cfg.batch, cfg.seqlen, cfg.nheads, cfg.ngroups)
    assert ssdi8.workspace_size(d) > 128 << 20
    import ctypes
    a = ssdi8.ScanArgs()
    assert ssdi8.lib().ssdi8_ssd_chunk_scan_noalloc(ctypes.byref(d), ctypes.byref(a), None) == \
        ssdi8.ERR_WORKSPACE
