"""The C ABI on the CPU (no GPU needed): the library loads and exports every function that
include/ssdi8.h declares, the binding's structs match the C layout, and every argument error
is reported by status code before anything is launched."""
import ctypes
import os
import re
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssdi8.h")


@pytest.fixture(scope="module")
def ssdi8():
    from paper_2608_21952_amd import ssdi8 as s
    if not os.path.exists(s.LIB_PATH):
        from paper_2608_21952_amd.build import build
        build()
    s.lib()
    return s


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(ssdi8_\w+)\s*\(", text, re.M)))


def test_every_declared_function_is_exported(ssdi8):
    names = declared_functions()
    assert {"ssdi8_quantize_act", "ssdi8_state_pass", "ssdi8_ssd_chunk_scan",
            "ssdi8_ssd_workspace_size", "ssdi8_status_string", "ssdi8_version"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", ssdi8.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (ssdi8_\w+)", out))
    assert set(names) <= exported, set(names) - exported
    for n in names:
        getattr(ssdi8.lib(), n)


def test_structs_match_the_header(ssdi8, tmp_path):
    fields = [f[0] for f in ssdi8.ScanArgs._fields_]
    src = tmp_path / "layout.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "ssdi8.h"', 'int main(void) {',
             'printf("%zu %zu\\n", sizeof(ssdi8_scan_args), sizeof(ssdi8_dims));']
    for f in fields:
        lines.append(f'printf("%zu\\n", offsetof(ssdi8_scan_args, {f}));')
    lines.append("return 0; }")
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    vals = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(ssdi8.ScanArgs)
    assert vals[1] == ctypes.sizeof(ssdi8.Dims)
    for f, off in zip(fields, vals[2:]):
        assert getattr(ssdi8.ScanArgs, f).offset == off, f


def test_fp16_struct_matches_the_header(ssdi8, tmp_path):
    fields = [f[0] for f in ssdi8.Fp16Args._fields_]
    src = tmp_path / "layout_f16.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "ssdi8.h"', 'int main(void) {',
             'printf("%zu\\n", sizeof(ssdi8_fp16_args));']
    for f in fields:
        lines.append(f'printf("%zu\\n", offsetof(ssdi8_fp16_args, {f}));')
    lines.append("return 0; }")
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout_f16"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    vals = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(ssdi8.Fp16Args)
    for f, off in zip(fields, vals[1:]):
        assert getattr(ssdi8.Fp16Args, f).offset == off, f


def test_fp16_argument_errors_and_workspace(ssdi8):
    L = ssdi8.lib()
    d = ssdi8.dims(2, 512, 8, 2)
    B, Lq, H, P, G, N, c = 2, 512, 8, 64, 2, 128, 2
    need = (2 * 2 * B * Lq * G * N + 2 * 4 * B * c * H * P * N + 4 * B * c * G * 36 * 1024
            + 4 * B * H * c)
    ws = ssdi8.fp16_workspace_size(d)
    assert need <= ws <= need + 6 * 256
    a = ssdi8.Fp16Args()
    for f in ("x", "dt", "A", "B", "C", "y", "workspace"):
        setattr(a, f, A16)
    a.x_dtype = a.y_dtype = a.bc_dtype = ssdi8.F16
    a.workspace_bytes = 1 << 40
    call = lambda dd, aa: L.ssdi8_ssd_chunk_scan_fp16(ctypes.byref(dd), ctypes.byref(aa), None)
    for f in ("x", "dt", "A", "B", "C", "y"):
        old = getattr(a, f)
        setattr(a, f, None)
        assert call(d, a) == ssdi8.ERR_NULL, f
        setattr(a, f, old)
    a.bc_dtype = 3
    assert call(d, a) == ssdi8.ERR_ARG
    a.bc_dtype = ssdi8.F16
    a.workspace_bytes = 16
    assert call(d, a) == ssdi8.ERR_WORKSPACE
    a.workspace_bytes = 1 << 40
    a.B = A16 + 8
    assert call(d, a) == ssdi8.ERR_ALIGN
    a.B = A16
    assert call(ssdi8.dims(2, 300, 8, 2), a) == ssdi8.ERR_SHAPE


def test_decode_struct_matches_the_header(ssdi8, tmp_path):
    fields = [f[0] for f in ssdi8.DecodeArgs._fields_]
    src = tmp_path / "layout_dec.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "ssdi8.h"', 'int main(void) {',
             'printf("%zu\\n", sizeof(ssdi8_decode_args));']
    for f in fields:
        lines.append(f'printf("%zu\\n", offsetof(ssdi8_decode_args, {f}));')
    lines.append("return 0; }")
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout_dec"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    vals = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(ssdi8.DecodeArgs)
    for f, off in zip(fields, vals[1:]):
        assert getattr(ssdi8.DecodeArgs, f).offset == off, f


def _decode_args(ssdi8, **over):
    a = ssdi8.DecodeArgs()
    for f in ("x", "dt", "A", "Bq", "Cq", "B_scale", "C_scale", "xs_scale", "state_scale",
              "cb_scale", "state_q", "y"):
        setattr(a, f, A16)
    a.x_dtype = a.y_dtype = ssdi8.F16
    a.decay_shift, a.shift_round, a.dt_softplus = 7, 1, 1
    for k, v in over.items():
        setattr(a, k, v)
    return a


def test_decode_argument_errors(ssdi8):
    dec = ssdi8.lib().ssdi8_decode_step

    def call(B=2, H=4, P=64, G=2, N=128, **over):
        return dec(B, H, P, G, N, ctypes.byref(_decode_args(ssdi8, **over)), None)
    assert dec(2, 4, 64, 2, 128, None, None) == ssdi8.ERR_NULL
    for f in ("x", "dt", "A", "Bq", "Cq", "B_scale", "C_scale", "xs_scale", "state_scale",
              "cb_scale", "state_q", "y"):
        assert call(**{f: None}) == ssdi8.ERR_NULL, f
    assert call(B=0, x=None) == ssdi8.OK                       # nothing to do
    assert call(B=-1) == ssdi8.ERR_SHAPE
    assert call(H=6, G=4) == ssdi8.ERR_SHAPE
    assert call(P=32) == ssdi8.ERR_UNSUPPORTED
    assert call(N=64) == ssdi8.ERR_UNSUPPORTED
    assert call(decay_shift=0) == ssdi8.ERR_ARG
    assert call(x_dtype=4) == ssdi8.ERR_ARG
    assert call(Bq=A16 + 4) == ssdi8.ERR_ALIGN
    assert call(state_q=A16 + 8) == ssdi8.ERR_ALIGN


def test_status_strings_and_version(ssdi8):
    for s in range(8):
        assert ssdi8.status_string(s)
    assert "unknown" in ssdi8.status_string(99)
    assert re.match(r"\d+\.\d+\.\d+", ssdi8.version())


def test_workspace_size(ssdi8):
    d = ssdi8.dims(4, 4096, 80, 1)
    B, L, H, P, G, N, Q = 4, 4096, 80, 64, 1, 128, 256
    c = L // Q
    # B_q^T and C_q copies, S_q and P_in, the 36 causal 32x32 blocks of CB_q, Q(Decay), and the
    # single-pass hand-off words: 64 ticket counters on lines of 32 words, the line of the wait
    # counter, one flag per item
    need = (2 * B * L * G * N + 2 * B * c * H * P * N + B * c * G * 36 * 32 * 32 + B * H * c * 2
            + 4 * (64 * 32 + 32 + B * H * c))
    ws = ssdi8.workspace_size(d)
    assert need <= ws <= need + 7 * 256
    assert ssdi8.workspace_size(ssdi8.dims(1, 300, 4, 1)) == 0          # L % chunk
    assert ssdi8.workspace_size(ssdi8.dims(1, 512, 6, 4)) == 0          # H % G
    assert ssdi8.workspace_size(ssdi8.dims(1, 512, 4, 1, headdim=32)) == 0


A16 = 0x10000          # fake, 16-byte aligned device addresses: never dereferenced on error paths


def _scan_args(ssdi8, **over):
    a = ssdi8.ScanArgs()
    for f in ("x", "dt", "A", "Bq", "Cq", "B_scale", "C_scale", "xs_scale", "state_scale",
              "cb_scale", "y", "workspace"):
        setattr(a, f, A16)
    a.x_dtype = a.y_dtype = ssdi8.F16
    a.decay_shift, a.shift_round, a.dt_softplus = 7, 1, 1
    a.workspace_bytes = 1 << 40
    for k, v in over.items():
        setattr(a, k, v)
    return a


def _scan(ssdi8, d, a):
    return ssdi8.lib().ssdi8_ssd_chunk_scan(ctypes.byref(d), ctypes.byref(a), None)


@pytest.mark.parametrize("field", ["x", "dt", "A", "Bq", "Cq", "B_scale", "C_scale", "xs_scale",
                                   "state_scale", "cb_scale", "y"])
def test_scan_null_pointer(ssdi8, field):
    assert _scan(ssdi8, ssdi8.dims(1, 512, 4, 1), _scan_args(ssdi8, **{field: None})) == \
        ssdi8.ERR_NULL


def test_scan_argument_errors(ssdi8):
    L = ssdi8.lib()
    ok = ssdi8.dims(1, 512, 4, 2)
    assert L.ssdi8_ssd_chunk_scan(None, ctypes.byref(_scan_args(ssdi8)), None) == ssdi8.ERR_NULL
    assert L.ssdi8_ssd_chunk_scan(ctypes.byref(ok), None, None) == ssdi8.ERR_NULL
    assert _scan(ssdi8, ssdi8.dims(1, 300, 4, 2), _scan_args(ssdi8)) == ssdi8.ERR_SHAPE
    assert _scan(ssdi8, ssdi8.dims(1, 512, 6, 4), _scan_args(ssdi8)) == ssdi8.ERR_SHAPE
    assert _scan(ssdi8, ssdi8.dims(-1, 512, 4, 2), _scan_args(ssdi8)) == ssdi8.ERR_SHAPE
    assert _scan(ssdi8, ssdi8.dims(1, 512, 4, 2, headdim=128), _scan_args(ssdi8)) == \
        ssdi8.ERR_UNSUPPORTED
    assert _scan(ssdi8, ssdi8.dims(1, 512, 4, 2, dstate=64), _scan_args(ssdi8)) == \
        ssdi8.ERR_UNSUPPORTED
    assert _scan(ssdi8, ssdi8.dims(1, 1024, 4, 2, chunk=128), _scan_args(ssdi8)) == \
        ssdi8.ERR_UNSUPPORTED
    assert _scan(ssdi8, ok, _scan_args(ssdi8, decay_shift=0)) == ssdi8.ERR_ARG
    assert _scan(ssdi8, ok, _scan_args(ssdi8, decay_shift=15)) == ssdi8.ERR_ARG
    assert _scan(ssdi8, ok, _scan_args(ssdi8, x_dtype=5)) == ssdi8.ERR_ARG
    assert _scan(ssdi8, ok, _scan_args(ssdi8, x=A16 + 8)) == ssdi8.ERR_ALIGN
    assert _scan(ssdi8, ok, _scan_args(ssdi8, state_q=A16 + 4)) == ssdi8.ERR_ALIGN
    assert _scan(ssdi8, ok, _scan_args(ssdi8, hand_off_timeouts=A16 + 2)) == ssdi8.ERR_ALIGN
    assert _scan(ssdi8, ok, _scan_args(ssdi8, workspace_bytes=16)) == ssdi8.ERR_WORKSPACE
    assert _scan(ssdi8, ok, _scan_args(ssdi8, workspace=None)) == ssdi8.ERR_WORKSPACE
    ev = (ctypes.c_void_p * 5)(A16, A16, None, A16, A16)
    assert _scan(ssdi8, ok, _scan_args(ssdi8, stage_events=ctypes.cast(ev, ctypes.c_void_p))) == \
        ssdi8.ERR_NULL


def test_quantize_argument_errors(ssdi8):
    q = ssdi8.lib().ssdi8_quantize_act
    assert q(A16, 1, 2, 8, 1, 128, 1, None, 0, A16, None) == ssdi8.ERR_NULL
    assert q(None, 1, 2, 8, 1, 128, 1, A16, 0, A16, None) == ssdi8.ERR_NULL
    assert q(A16, 3, 2, 8, 1, 128, 1, A16, 0, A16, None) == ssdi8.ERR_ARG
    assert q(A16, 1, 2, 8, 1, 128, 7, A16, 0, A16, None) == ssdi8.ERR_ARG
    assert q(A16, 1, -2, 8, 1, 128, 1, A16, 0, A16, None) == ssdi8.ERR_SHAPE
    assert q(A16, 1, 2, 8, 0, 128, 1, A16, 0, A16, None) == ssdi8.ERR_SHAPE
    assert q(A16 + 2, 1, 2, 8, 1, 128, 1, A16, 0, A16, None) == ssdi8.ERR_ALIGN
    assert q(A16, 1, 2, 8, 64, 256, 2, A16, 1, A16, None) == ssdi8.ERR_UNSUPPORTED


def test_state_pass_argument_errors(ssdi8):
    sp = ssdi8.lib().ssdi8_state_pass
    args = dict(sq=A16, qd=A16, shift=7, rnd=1, init=None, pin=A16, fq=None, fs=None, ss=None)

    def call(**kw):
        a = dict(args)
        a.update(kw)
        return sp(a["sq"], a["qd"], a["shift"], a["rnd"], a["init"], a["pin"], a["fq"],
                  a["fs"], a["ss"], 1, 4, 2, 64, 128, None)
    assert call(sq=None) == ssdi8.ERR_NULL
    assert call(pin=None) == ssdi8.ERR_NULL
    assert call(fs=A16) == ssdi8.ERR_NULL            # fp32 state needs the state steps
    assert call(shift=0) == ssdi8.ERR_ARG
    assert call(qd=A16 + 1) == ssdi8.ERR_ALIGN
    assert sp(A16, A16, 7, 1, None, A16, None, None, None, 1, 4, 2, 64, 126, None) == \
        ssdi8.ERR_UNSUPPORTED


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


@pytest.mark.parametrize("name,heads", [("mamba2-8b-g8", 16), ("mamba2-130m", 4)])
def test_bench_cpu_baseline_samples_any_group_count(name, heads):
    """The oracle's timed sample takes whole heads of group 0 when it cannot take every head."""
    sys.path.insert(0, ROOT)
    import bench
    from oracle import calibrate
    from paper_2608_21952_amd import synth
    cfg = synth.CONFIGS[name].scaled(name="t", batch=2, seqlen=512, nheads=heads)
    inp, cal = synth.draw(cfg, 1), synth.draw(cfg, 2)
    sc = calibrate.calibrate(cal["x"], cal["dt_raw"], cal["A"], cal["B"], cal["C"], cal["D"],
                             chunk=cfg.chunk)
    part = bench.cpu_baseline(cfg, inp, sc, 1e-6)
    assert part["kind"] == "oracle" and part["value"] > 0 and "heads 0.." in part["sample"]
    whole = bench.cpu_baseline(cfg, inp, sc, 1e6)
    assert whole["sample"].startswith("the whole workload")


def test_bench_head_sample_keeps_whole_groups():
    sys.path.insert(0, ROOT)
    import bench
    assert [bench.sample_heads(n, 128, 8) for n in (1, 15, 16, 17, 40, 127, 128, 300)] == \
        [1, 15, 16, 16, 32, 112, 128, 128]
    assert [bench.sample_heads(n, 80, 1) for n in (1, 79, 80)] == [1, 79, 80]


def test_calib_struct_matches_the_header(ssdi8, tmp_path):
    fields = [f[0] for f in ssdi8.CalibArgs._fields_]
    src = tmp_path / "layout_cal.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "ssdi8.h"', 'int main(void) {',
             'printf("%zu\\n", sizeof(ssdi8_calib_args));']
    for f in fields:
        lines.append(f'printf("%zu\\n", offsetof(ssdi8_calib_args, {f}));')
    lines.append("return 0; }")
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout_cal"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    vals = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                           check=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(ssdi8.CalibArgs)
    for f, off in zip(fields, vals[1:]):
        assert getattr(ssdi8.CalibArgs, f).offset == off, f


def test_calib_argument_errors_and_workspace(ssdi8):
    L = ssdi8.lib()
    d = ssdi8.dims(2, 512, 8, 2)
    B, Lq, H, P, G, N = 2, 512, 8, 64, 2, 128
    ws = ssdi8.calibrate_workspace_size(d)
    parts = (ssdi8.fp16_workspace_size(d) + ssdi8.workspace_size(d) + 2 * B * Lq * G * N
             + 2 * 4 * B * Lq * H * P + 8 * B * H * 2 + 4 * (2 * H * P + G) + 8 * H * 64 * P)
    assert parts <= ws <= parts + 9 * 256
    assert ssdi8.calibrate_workspace_size(ssdi8.dims(0, 512, 8, 2)) == 0
    a = ssdi8.CalibArgs()
    for f in ("x", "dt", "A", "B", "C", "B_scale", "C_scale", "xs_scale", "state_scale",
              "cb_scale", "corr", "workspace"):
        setattr(a, f, A16)
    a.x_dtype = a.bc_dtype = ssdi8.F16
    a.eta, a.decay_shift, a.shift_round = 0.15, 7, 1
    a.workspace_bytes = 1 << 40
    call = lambda dd, aa: L.ssdi8_calibrate(ctypes.byref(dd), ctypes.byref(aa), None)
    for f in ("x", "dt", "A", "B", "C", "B_scale", "C_scale", "xs_scale", "state_scale",
              "cb_scale", "corr"):
        old = getattr(a, f)
        setattr(a, f, None)
        assert call(d, a) == ssdi8.ERR_NULL, f
        setattr(a, f, old)
    a.decay_shift = 15
    assert call(d, a) == ssdi8.ERR_ARG
    a.decay_shift = 7
    a.eta = float("nan")
    assert call(d, a) == ssdi8.ERR_ARG
    a.eta = 0.15
    a.workspace_bytes = ws - 1
    assert call(d, a) == ssdi8.ERR_WORKSPACE
    a.workspace_bytes = 1 << 40
    a.corr = A16 + 2
    assert call(d, a) == ssdi8.ERR_ALIGN
    a.corr = A16
    assert call(ssdi8.dims(0, 512, 8, 2), a) == ssdi8.ERR_SHAPE
    assert call(ssdi8.dims(2, 300, 8, 2), a) == ssdi8.ERR_SHAPE


def test_single_pass_selection(ssdi8):
    """The automatic choice between the single pass and the separate kernels (host only)."""
    import torch
    f16, f32 = torch.float16, torch.float32
    use = lambda dd, *a, **k: ssdi8.uses_single_pass(dd, *a, **k)
    assert use(ssdi8.dims(8, 2048, 24, 1), f16)                # 192 sequences of 8 chunks
    assert use(ssdi8.dims(4, 2048, 24, 1), f16)                # 96 sequences of 8 chunks
    assert use(ssdi8.dims(3, 1024, 24, 1), f16)                # 72 sequences of 4 chunks
    assert not use(ssdi8.dims(3, 768, 24, 1), f16)             # 72 sequences of 3 chunks
    assert not use(ssdi8.dims(8, 512, 24, 1), f16)             # 2 chunks
    assert not use(ssdi8.dims(2, 4096, 24, 1), f16)            # 48 sequences of 16 chunks
    assert use(ssdi8.dims(2, 8192, 24, 1), f16)                # 48 sequences of 32 chunks
    assert not use(ssdi8.dims(1, 65536, 24, 1), f16)           # 24 sequences: chain-bound
    assert use(ssdi8.dims(4, 4096, 80, 1), f16)                # 16 chunks, 320 sequences
    assert use(ssdi8.dims(2, 8192, 128, 8), f16)
    assert use(ssdi8.dims(1, 65536, 80, 1), f16)               # 80 sequences of 256 chunks
    assert use(ssdi8.dims(1, 4096, 96, 1), f16)                # 96 sequences of 16 chunks
    assert not use(ssdi8.dims(1, 4096, 40, 1), f16)            # 40 sequences of 16 chunks
    assert use(ssdi8.dims(8, 2048, 24, 1), f16, "single")
    assert not use(ssdi8.dims(4, 4096, 80, 1), f16, "separate")
    assert not use(ssdi8.dims(4, 4096, 80, 1), f32, "single")  # fp32 x: separate kernels
    assert not use(ssdi8.dims(4, 4096, 80, 1), f16, "single", taps=("state_q",))
    assert not use(ssdi8.dims(4, 4096, 80, 1), f16, "single", taps=("dt_post",))
    # ChunkBMM's taps and the entering states are available from the single pass
    assert use(ssdi8.dims(4, 4096, 80, 1), f16, "single", taps=("cb_q",))
    assert use(ssdi8.dims(4, 4096, 80, 1), f16, "single", taps=("state_in_q",))
    assert use(ssdi8.dims(4, 4096, 80, 1), f16, taps=("state_in_q",))
    assert not use(ssdi8.dims(4, 300, 80, 1), f16, "single")   # invalid sizes


def test_scan_path_out_of_range(ssdi8):
    L = ssdi8.lib()
    d = ssdi8.dims(2, 512, 8, 2)
    a = ssdi8.ScanArgs()
    for f in ("x", "dt", "A", "Bq", "Cq", "B_scale", "C_scale", "xs_scale", "state_scale",
              "cb_scale", "y", "workspace"):
        setattr(a, f, A16)
    a.x_dtype = a.y_dtype = ssdi8.F16
    a.decay_shift, a.workspace_bytes = 7, 1 << 40
    a.path = 3
    assert L.ssdi8_ssd_chunk_scan(ctypes.byref(d), ctypes.byref(a), None) == ssdi8.ERR_ARG


def test_mfma_probe_argument_errors(ssdi8):
    L = ssdi8.lib()
    ops = ctypes.c_int64()
    assert L.ssdi8_mfma_probe(2, 10, 4, A16, ctypes.byref(ops), None) == ssdi8.ERR_ARG
    assert L.ssdi8_mfma_probe(0, 0, 4, A16, ctypes.byref(ops), None) == ssdi8.ERR_ARG
    assert L.ssdi8_mfma_probe(0, 10, 0, A16, ctypes.byref(ops), None) == ssdi8.ERR_ARG
    assert L.ssdi8_mfma_probe(0, 10, 70000, A16, ctypes.byref(ops), None) == ssdi8.ERR_ARG
    assert L.ssdi8_mfma_probe(0, 10, 4, None, ctypes.byref(ops), None) == ssdi8.ERR_NULL
    assert L.ssdi8_mfma_probe(1, 10, 4, A16 + 2, ctypes.byref(ops), None) == ssdi8.ERR_ALIGN


def test_scan_unquantized_bc_arguments(ssdi8):
    L = ssdi8.lib()
    d = ssdi8.dims(2, 512, 8, 2)
    a = ssdi8.ScanArgs()
    for f in ("x", "dt", "A", "B", "C", "B_scale", "C_scale", "xs_scale", "state_scale",
              "cb_scale", "y", "workspace"):
        setattr(a, f, A16)
    a.x_dtype = a.y_dtype = a.bc_dtype = ssdi8.F16
    a.decay_shift, a.workspace_bytes = 7, 1 << 40
    call = lambda: L.ssdi8_ssd_chunk_scan(ctypes.byref(d), ctypes.byref(a), None)
    a.Bq = A16                        # both forms at once
    assert call() == ssdi8.ERR_ARG
    a.Bq = None
    a.bc_dtype = 5
    assert call() == ssdi8.ERR_ARG
    a.bc_dtype = ssdi8.F16
    a.C = None
    assert call() == ssdi8.ERR_NULL
    a.C = A16 + 4
    assert call() == ssdi8.ERR_ALIGN


def test_traffic_source_hash_ignores_comments_only():
    """The stored HBM traffic of a kernel stays valid across comment edits, not code edits."""
    import bench
    code = "int f() { return 1; } // one\n/* two\n   lines */ int g;\n"
    assert bench._code_only(code) == bench._code_only("int f() {  return 1; }\n\nint g;")
    assert bench._code_only(code) != bench._code_only("int f() { return 2; }\nint g;")
    assert bench.kernel_source_sha256("single_pass") is not None
