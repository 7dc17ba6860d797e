"""Shared helpers of the parity tests: seeded inputs, oracle-side calibration, GPU calls through
the C ABI binding, and the stage-isolated comparisons (the oracle re-runs each integer stage on
the GPU's own inputs to that stage, so a mismatch names the stage that produced it)."""
from __future__ import annotations

import os
import sys
from typing import Dict, Iterable, Optional, Tuple

import numpy as np

from oracle import calibrate as ocal
from oracle import exact as oex
from oracle import int8 as oq
from paper_2608_21952_amd import synth

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
CALIB_DIR = os.path.join(GOLD, "calib")

# y tolerance (floating-point output): max |dy| / max |y_oracle| and relative L2.
TOL_MAXABS = 1e-2
TOL_RELL2 = 1e-3

SCALE_KEYS = ("alpha_B", "alpha_C", "alpha_Xs", "alpha_S", "alpha_CB", "corr")


def say(*a) -> None:
    print(*a, flush=True)
    sys.stdout.flush()


def calibration(cfg: synth.SSDConfig) -> Dict[str, np.ndarray]:
    """Stored scales for a named workload (written by tests/golden/make_calibration.py from the
    oracle), or a fresh oracle calibration on the s = 2 draw for ad-hoc shapes."""
    path = os.path.join(CALIB_DIR, cfg.name + ".npz")
    if cfg.name in synth.CONFIGS and synth.CONFIGS[cfg.name] == cfg and os.path.exists(path):
        with np.load(path, allow_pickle=False) as z:
            return {k: z[k] for k in SCALE_KEYS}
    d = synth.draw(cfg, 2)
    return ocal.calibrate(d["x"], d["dt_raw"], d["A"], d["B"], d["C"], d["D"],
                          chunk=cfg.chunk, xs_per_head=cfg.xs_per_head)


def rel_errors(y_gpu, y_ref) -> Tuple[float, float]:
    g = np.asarray(y_gpu, np.float64)
    r = np.asarray(y_ref, np.float64)
    scale = max(np.abs(r).max(), 1e-30)
    maxabs = float(np.abs(g - r).max()) / scale
    rel = float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30))
    return maxabs, rel


def assert_equal(gpu, ref, what: str) -> None:
    """Bit-exact comparison that names the stage and shows where it differs."""
    gpu = np.asarray(gpu)
    ref = np.asarray(ref)
    assert gpu.shape == ref.shape, f"{what}: shape {gpu.shape} vs {ref.shape}"
    bad = gpu != ref
    if bad.any():
        idx = np.argwhere(bad)
        first = [(tuple(int(v) for v in i), gpu[tuple(i)].item(), ref[tuple(i)].item())
                 for i in idx[:8]]
        raise AssertionError(f"{what} mismatch: {int(bad.sum())} of {bad.size} differ; "
                             f"first (index, gpu, oracle): {first}")


def assert_close(y_gpu, y_ref, what="y") -> Tuple[float, float]:
    maxabs, rel = rel_errors(y_gpu, y_ref)
    say(f"  {what}: max|d|/max|ref| = {maxabs:.3e}  relL2 = {rel:.3e}")
    assert maxabs <= TOL_MAXABS, f"{what} max-abs error {maxabs:.3e} > {TOL_MAXABS}"
    assert rel <= TOL_RELL2, f"{what} relative L2 error {rel:.3e} > {TOL_RELL2}"
    return maxabs, rel


# ------------------------------------------------------------------------------ GPU side
def dev(a, torch):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run_layer(torch, ssdi8, inp: Dict[str, np.ndarray], sc: Dict[str, np.ndarray], *,
              taps: Iterable[str] = (), dt_softplus: bool = True, init_q=None,
              decay_shift: int = 7, shift_round: bool = True, c_per_token: bool = False,
              use_D: bool = True, use_corr: bool = True, y_dtype=None, keep_on_device=False,
              path: str = "auto", workspace=None):
    """Quantize B, C with the static steps (ssdi8_quantize_act) and run ssdi8_ssd_chunk_scan.
    Returns numpy arrays (or device tensors) of y, final states, Bq, Cq, the taps and
    `hand_off_timeouts` (the count of single-pass waits that ran out)."""
    x = dev(inp["x"], torch)
    dt = dev(inp["dt_raw"], torch)
    B = dev(inp["B"], torch)
    C = dev(inp["C"], torch)
    f32 = lambda v: dev(np.asarray(v, np.float32), torch)
    aB, aXs, aS, aCB = f32(sc["alpha_B"]), f32(sc["alpha_Xs"]), f32(sc["alpha_S"]), f32(sc["alpha_CB"])
    Bq, _ = ssdi8.quantize_act(B, "group", aB)
    if c_per_token:
        Cq, aC = ssdi8.quantize_act(C, "token")
        aC = aC.view(C.shape[0], C.shape[1], C.shape[2])
    else:
        aC = f32(sc["alpha_C"])
        Cq, _ = ssdi8.quantize_act(C, "group", aC)
    out = ssdi8.ssd_chunk_scan(
        x, dt, f32(inp["A"]), Bq, Cq, aB, aC, aXs, aS, aCB,
        D=f32(inp["D"]) if use_D else None, corr=f32(sc["corr"]) if use_corr else None,
        dt_softplus=dt_softplus, decay_shift=decay_shift, shift_round=shift_round,
        init_state_q=None if init_q is None else dev(init_q, torch), taps=taps,
        y_dtype=y_dtype, path=path, workspace=workspace,
        hand_off_timeouts=torch.full((1,), -1, dtype=torch.int32, device="cuda"))
    out["Bq"], out["Cq"] = Bq, Cq
    if c_per_token:
        out["C_scale"] = aC
    torch.cuda.synchronize()
    if keep_on_device:
        return out
    return {k: v.cpu().numpy() for k, v in out.items()}


# ------------------------------------------------------------------------------ comparisons
def oracle_scales(sc, c_scale=None):
    s = {k: sc[k] for k in ("alpha_B", "alpha_C", "alpha_Xs", "alpha_S", "alpha_CB")}
    if c_scale is not None:
        s["alpha_C"] = c_scale
    return s


def check_slab(g: Dict[str, np.ndarray], inp, sc, b: int, h: int, cfg_chunk: int, *,
               dt_softplus=True, k=7, shift_round=True, init_q=None, c_scale=None,
               use_D=True, use_corr=True, out_dtype=np.float16, check_end_to_end=True):
    """Compare one (batch, head) slab of a GPU run with the oracle, stage by stage.  `g` holds
    the GPU outputs (numpy) incl. the taps xs_q, state_i32, state_q, decay_q, state_in_q,
    cb_i32, cb_q, scan1_i32 if they were requested."""
    H = inp["x"].shape[2]
    G = inp["B"].shape[2]
    gi = int(oex.head_group(H, G)[h])
    Q = cfg_chunk
    scs = oracle_scales(sc, c_scale)
    s = oq.scales_for_head(scs, h, gi, b, inp["x"].shape[3])
    A_h = np.float32(inp["A"][h])
    dt32 = oq.dt_post(inp["dt_raw"][b, :, h], dt_softplus)
    Bq_g, Cq_g = g["Bq"][b, :, gi], g["Cq"][b, :, gi]
    # ChunkCumsum + Q(Decay)
    cum = oq.chunk_cumsum(dt32, A_h, Q, k)
    fragile = oq.fragile_tokens(inp["dt_raw"][b, :, h], A_h, Q, dt_softplus, k)
    if "decay_q" in g:
        bad = g["decay_q"][b, h] != cum["qd"]
        badc = fragile.reshape(-1, Q).any(axis=1)
        assert np.all(~bad | badc), f"Q(Decay) mismatch at chunks {np.nonzero(bad)[0]}"
    # ChunkState: X_q end-to-end (fragile tokens excepted), then S32 and S_q stage-isolated
    if "xs_q" in g:
        st = oq.chunk_state(inp["x"][b, :, h], cum["lut"], Bq_g, s["alpha_xs"], s["alpha_B"],
                            s["alpha_S"])
        xq = g["xs_q"][b, :, h]
        mism = np.any(xq != st["Xq"], axis=1)
        assert np.all(~mism | fragile), f"X_q mismatch at tokens {np.nonzero(mism & ~fragile)[0][:10]}"
        if mism.any():
            say(f"  X_q: {int(mism.sum())} fragile tokens differ")
        if "state_i32" in g:
            nc = xq.shape[0] // Q
            s32 = oq._int_matmul(np.swapaxes(xq.reshape(nc, Q, -1), 1, 2),
                                 Bq_g.reshape(nc, Q, -1))
            assert_equal(g["state_i32"][b, :, h], s32, "State_INT32")
            if "state_q" in g:
                ms = oq.multiplier(s["alpha_xs"], s["alpha_B"], s["alpha_S"])
                sq = oq.requant(g["state_i32"][b, :, h], ms[None, :, None])
                assert_equal(g["state_q"][b, :, h], sq, "State_INT8")
    # StatePassing, stage-isolated on the GPU's S_q and q_d
    if "state_in_q" in g and "state_q" in g and "decay_q" in g:
        init = None if init_q is None else init_q[b, h]
        pin, fin = oq.state_pass(g["state_q"][b, :, h], g["decay_q"][b, h], init, k, shift_round)
        assert_equal(g["state_in_q"][b, :, h], pin, "P_in")
        assert_equal(g["final_state_q"][b, h], fin, "final_q")
        fs = fin.astype(np.float32) * np.asarray(sc["alpha_S"], np.float32)[h][:, None]
        assert_equal(g["final_state"][b, h], fs, "final fp32 state")
    # ChunkBMM, stage-isolated on the GPU's B_q, C_q
    if "cb_i32" in g:
        cb = oq.chunk_bmm(Cq_g, Bq_g, s["alpha_C"], s["alpha_B"], s["alpha_CB"], Q)
        assert_equal(g["cb_i32"][b, :, gi], cb["CB32"], "CB_INT32")
        if "cb_q" in g:
            assert_equal(g["cb_q"][b, :, gi], cb["CBq"], "CB_INT8")
    # ChunkScan1 product, stage-isolated on the GPU's C_q and P_in
    if "scan1_i32" in g and "state_in_q" in g:
        nc = Cq_g.shape[0] // Q
        y1 = oq._int_matmul(Cq_g.reshape(nc, Q, -1),
                            np.swapaxes(g["state_in_q"][b, :, h], 1, 2)).reshape(-1, g["state_in_q"].shape[3])
        assert_equal(g["scan1_i32"][b, :, h], y1, "ChunkScan1 INT32")
    D_h = np.float32(inp["D"][h]) if use_D else np.float32(0)
    corr_h = np.asarray(sc["corr"], np.float32)[h] if use_corr else np.zeros(inp["x"].shape[3], np.float32)
    # output, stage-isolated: oracle ChunkScan on the GPU's P_in and CB_q
    if "state_in_q" in g and "cb_q" in g:
        scan = oq.chunk_scan(Cq_g, g["state_in_q"][b, :, h], g["cb_q"][b, :, gi], cum,
                             inp["x"][b, :, h], s["alpha_C"], s["alpha_S"], s["alpha_CB"], D_h,
                             corr_h, out_dtype)
        assert_close(g["y"][b, :, h], scan["y"], f"y[b={b},h={h}] (stage-isolated)")
    if check_end_to_end:
        init = None if init_q is None else init_q[b, h]
        Bo, _ = oq.quantize_act(inp["B"][b:b + 1, :, gi:gi + 1], "group",
                                np.asarray(sc["alpha_B"], np.float32)[gi:gi + 1])
        if c_scale is not None:       # per-token C steps: the oracle derives its own
            Co, aCo = oq.quantize_act(inp["C"][b:b + 1, :, gi:gi + 1], "token")
            assert_equal(s["alpha_C"], aCo[0, :, 0], "per-token C steps")
        else:
            Co, _ = oq.quantize_act(inp["C"][b:b + 1, :, gi:gi + 1], "group",
                                    np.asarray(sc["alpha_C"], np.float32)[gi:gi + 1])
        assert_equal(Bq_g, Bo[0, :, 0], "B_q")
        assert_equal(Cq_g, Co[0, :, 0], "C_q")
        ref = oq.ssdi8_slab(inp["x"][b, :, h], dt32, A_h, Bo[0, :, 0], Co[0, :, 0], D_h, corr_h,
                            s, Q, k, shift_round, init, out_dtype)
        assert_close(g["y"][b, :, h], ref["y"], f"y[b={b},h={h}] (end-to-end)")
        return ref
    return None
