#!/usr/bin/env python3
"""Throughput of the SSDi8 INT8 SSD chunk scan (one SSD layer) on one MI355X.

A step is one whole layer on one batch of synthetic Mamba-2-shaped input already resident in
HBM: ssdi8_ssd_chunk_scan on the unquantized B and C (ChunkBMM quantizes them per group with the
static steps, then ChunkCumsum + ChunkState, StatePassing, ChunkScan 1+2 with the D skip and the
correction; --separate-quant times ssdi8_quantize_act x 2 + the scan on B_q, C_q instead).
Scales are static (calibrated offline by the CPU oracle; stored in tests/golden/calib).

Prints ONE JSON line: tokens/s per layer, ms/step, the roofline of the dominant kernel measured
live with HIP events on the launch stream, per-module times, and the CPU oracle timed on a
bounded sample of the same workload on this host's cores.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, published
INT8_PEAK_TOPS = 5000.0         # MI355X dense int8 MFMA, published
FP16_PEAK_TFLOPS = 2500.0       # MI355X dense fp16 MFMA, published
MODULES = ("chunk_bmm", "chunk_state", "state_pass", "chunk_scan")
# the single pass (fp16 x): ChunkState + StatePassing + ChunkScan in one kernel after ChunkBMM
SINGLE = ("chunk_bmm", "single_pass")
SOURCE = {"single_pass": "chunk_scan"}      # kernel -> source file of its HIP code
# headers every kernel source compiles in: a change to them is a change to the kernel
KERNEL_HEADERS = ("common.hpp", "exact_sum.hpp", "frag.hpp", "launch.hpp")


def _code_only(text: str) -> str:
    """The source without its comments and blank space, so that a comment edit does not count
    as a change of the kernel (none of these sources has // or /* inside a string literal)."""
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(" ".join(line.split()) for line in text.splitlines() if line.strip())


def kernel_source_sha256(kernel: str):
    """sha256 over the code of the kernel's .hip source followed by the shared headers, comments
    and blank space left out (None if one is missing)."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2608_21952_amd", "csrc")
    h = hashlib.sha256()
    for name in (f"{SOURCE.get(kernel, kernel)}.hip",) + KERNEL_HEADERS:
        path = os.path.join(csrc, name)
        if not os.path.exists(path):
            return None
        with open(path, encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def algorithmic_bytes(cfg, quant_in_bmm=False):
    """Minimum HBM bytes each kernel must move for its inputs and outputs (per launch); with
    quant_in_bmm ChunkBMM reads the unquantized B and C."""
    B, L, H, P, G, N, Q = (cfg.batch, cfg.seqlen, cfg.nheads, cfg.headdim, cfg.ngroups,
                           cfg.dstate, cfg.chunk)
    T, c = B * L, L // Q
    sx = 2 if cfg.dtype == "fp16" else 4
    states = B * c * H * P * N                       # one int8 state tensor (B,c,H,P,N)
    cb_causal = B * c * G * Q * (Q + 1) // 2
    return {
        "quantize_B": T * G * N * (sx + 1),
        "quantize_C": T * G * N * (sx + 1),
        "chunk_bmm": 2 * T * G * N * (sx if quant_in_bmm else 1) + cb_causal,
        "chunk_state": T * H * P * sx + T * H * 4 + T * G * N + states + B * H * c * 2,
        "state_pass": 2 * states + B * H * c * 2 + B * H * P * N * 5,
        "chunk_scan": 2 * T * H * P * sx + T * H * 4 + T * G * N + states + cb_causal,
        # x in, y out, dt, B_q^T and C_q (per group), CB_q and the final state (int8 + fp32);
        # the states handed from chunk to chunk are overhead (single_pass_overhead)
        "single_pass": (2 * T * H * P * sx + T * H * 4 + 2 * T * G * N + cb_causal
                        + B * H * P * N * 5),
    }


def single_pass_overhead(cfg):
    """Bytes the single pass moves beyond the minimum of its inputs and outputs: the int8 state
    entering each chunk after the first, written by the chunk before it and read once."""
    B, L, H, P, N, Q = cfg.batch, cfg.seqlen, cfg.nheads, cfg.headdim, cfg.dstate, cfg.chunk
    c = L // Q
    return {"hand_off_states": 2 * B * max(c - 1, 0) * H * P * N}


def algorithmic_ops(cfg):
    """Algorithmic MFMA work per launch (multiply + add = 2 ops), causal products counted over
    i <= j only: {kernel: (int8 ops, fp16 flops)}."""
    B, L, H, P, G, N, Q = (cfg.batch, cfg.seqlen, cfg.nheads, cfg.headdim, cfg.ngroups,
                           cfg.dstate, cfg.chunk)
    c = L // Q
    pairs = Q * (Q + 1) // 2
    return {
        "chunk_bmm": (2 * B * c * G * pairs * N, 0),
        "chunk_state": (2 * B * c * H * Q * P * N, 0),
        "chunk_scan": (2 * B * c * H * Q * N * P, 2 * B * c * H * pairs * P),
        "single_pass": (2 * B * c * H * Q * P * N + 2 * B * c * H * Q * N * P,
                        2 * B * c * H * pairs * P),
    }


def layer_min_bytes(cfg):
    """Layer-level minimum, per token: x in and y out (H P elements each), dt (4 H bytes), B and C
    at the input width (2 G N elements); plus the final state (int8 and fp32, 5 B H P N)."""
    B, L, H, P, G, N = cfg.batch, cfg.seqlen, cfg.nheads, cfg.headdim, cfg.ngroups, cfg.dstate
    sx = 2 if cfg.dtype == "fp16" else 4
    T = B * L
    return 2 * T * H * P * sx + T * H * 4 + 2 * T * G * N * sx + B * H * P * N * 5


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary (each counter scaled by what it reads for a plain copy of known size), or None when
    there is none or the kernel's source or a shared header changed since the counters were
    taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    digest = kernel_source_sha256(kernel)
    if not os.path.exists(path) or digest is None:
        return None
    with open(path) as f:
        rec = json.load(f)
    if digest != rec.get("source_sha256"):
        return None
    return rec.get("bytes_per_launch")


def sample_heads(nh: int, nheads: int, ngroups: int) -> int:
    """The head count of the oracle's sample nearest below `nh` that keeps the head-to-group
    map: all heads, heads of group 0 only, or whole groups."""
    hpg = nheads // ngroups
    if nh >= nheads:
        return nheads
    return nh if nh <= hpg else nh - nh % hpg


def cpu_baseline(cfg, inp, sc, budget_s: float):
    """The CPU oracle as it stands, timed on a bounded sample of the workload: the first `nh`
    heads of the first `nb` batch elements (all chunks), sized from pilots to about `budget_s`
    seconds; the whole workload when it fits."""
    import numpy as np
    import threadpoolctl
    from oracle import int8

    def run(nb, nh):
        # a head sample is the heads of group 0 or of whole groups 0 .. ng-1, with their B, C, steps
        ng = cfg.ngroups if nh == cfg.nheads else -(-nh // hpg)
        t = time.perf_counter()
        int8.ssdi8_forward(inp["x"][:nb, :, :nh], inp["dt_raw"][:nb, :, :nh], inp["A"][:nh],
                           inp["B"][:nb, :, :ng], inp["C"][:nb, :, :ng], inp["D"][:nh],
                           sc["corr"][:nh],
                           {"alpha_B": sc["alpha_B"][:ng], "alpha_C": sc["alpha_C"][:ng],
                            "alpha_Xs": sc["alpha_Xs"][:nh], "alpha_S": sc["alpha_S"][:nh],
                            "alpha_CB": sc["alpha_CB"][:ng]},
                           chunk=cfg.chunk, want=("y",))
        return time.perf_counter() - t

    G = cfg.ngroups
    hpg = cfg.nheads // G
    pilot = run(1, 1)
    nh = int(max(1, min(cfg.nheads, budget_s / max(pilot, 1e-3))))
    nb = 1
    nh = sample_heads(nh, cfg.nheads, G)
    if nh == cfg.nheads:
        one = run(1, nh)
        nb = int(max(1, min(cfg.batch, budget_s / max(one, 1e-3))))
    t = run(nb, nh)
    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] or [1])
    tokens = nb * cfg.seqlen * nh / cfg.nheads   # layer-tokens: a token carries all H heads
    whole = nb == cfg.batch and nh == cfg.nheads
    what = ("the whole workload" if whole else
            f"batch elements 0..{nb - 1} of {cfg.batch}, heads 0..{nh - 1} of {cfg.nheads}")
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": tokens / t, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": model,
            "sample": f"{what}, {cfg.seqlen} tokens each ({t:.1f} s; tokens/s counted as layer "
                      f"tokens = token-heads / {cfg.nheads})",
            "seconds": round(t, 2), "host_cpus": len(os.sched_getaffinity(0))}


def measured_peaks(torch, ssdi8):
    """On-box peaks: a 1 GiB device-to-device copy (bytes read + written per second) and the
    MFMA probe loops (int8, fp16), best of a few runs."""
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    best = 0.0
    for _ in range(4):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        best = max(best, 2 * n / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del src, dst
    return {"hbm_copy_GBps": round(best, 1),
            "int8_mfma_TOPS": round(ssdi8.mfma_peak("int8") / 1e12, 1),
            "fp16_mfma_TFLOPS": round(ssdi8.mfma_peak("fp16") / 1e12, 1),
            "how": "1 GiB device copy (read + write bytes); 1024 workgroups x 4 waves x 4 "
                   "independent MFMA chains on register operands (ssdi8_mfma_probe)"}


def keep_busy(graph, ms_step, seconds=0.05):
    """Replay the captured step for about `seconds` of GPU time without waiting for it, so that
    the host has queued the eager steps that follow before the GPU reaches them (it queues one
    faster than the GPU runs one) and the GPU meanwhile runs real work at steady clocks (a spin
    kernel would let them drop): events between those eager kernels then time GPU execution."""
    for _ in range(max(1, int(seconds * 1e3 / max(ms_step, 1e-3)))):
        graph.replay()


def time_fp16(torch, ssdi8, cfg, x, dt, A, Bf, Cf, D, K, W):
    """The unquantized FP16 SSD layer on the same inputs (ssdi8_ssd_chunk_scan_fp16): K replays
    of one captured graph for the step time, then K eager steps with stage events."""
    ws = torch.empty(max(ssdi8.fp16_workspace_size(ssdi8.dims(cfg.batch, cfg.seqlen, cfg.nheads,
                                                               cfg.ngroups)), 1),
                     dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    ev = ssdi8.HipEvents(5 * max(K, 1))

    def step(k=None):
        ssdi8.ssd_chunk_scan_fp16(x, dt, A, Bf, Cf, D=D, workspace=ws, y=y, final_state=True,
                                  stage_events=None if k is None else ev.group(5 * k))
    for _ in range(W):
        step()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    graph.replay()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(K):
        graph.replay()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / K
    keep_busy(graph, ms)
    for k in range(K):
        step(k)
    torch.cuda.synchronize()
    names = ("chunk_bmm", "chunk_state", "state_pass", "chunk_scan")
    per = {n: sum(ev.elapsed_ms(5 * k + i, 5 * k + i + 1) for k in range(K)) / K * 1e3
           for i, n in enumerate(names)}
    ev.close()
    return {"ms_per_step": ms, "tokens_per_s": cfg.batch * cfg.seqlen / (ms * 1e-3),
            "stages_us": {n: round(v, 2) for n, v in per.items()},
            "what": "the same layer unquantized: fp16 operands, fp32 states (Alg. 2)"}


def time_calibrate(torch, ssdi8, cfg, x, dt, A, Bf, Cf, D, K):
    """One static calibration of the workload on the device (ssdi8_calibrate: the steps of B, C,
    X_scaled, the states and C.B^T, then the FP16 and the INT8 layer and the mean correction),
    after one warmup call; K calls bracketed by events on the launch stream."""
    d = ssdi8.dims(cfg.batch, cfg.seqlen, cfg.nheads, cfg.ngroups)
    ws = torch.empty(max(ssdi8.calibrate_workspace_size(d), 1), dtype=torch.uint8, device="cuda")
    call = lambda: ssdi8.calibrate(x, dt, A, Bf, Cf, D=D, xs_per_head=cfg.xs_per_head,
                                   workspace=ws)
    call()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(K):
        call()
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / K
    return {"ms_per_call": round(ms, 3), "tokens_per_s": cfg.batch * cfg.seqlen / (ms * 1e-3),
            "calls": K, "workspace_MB": round(ws.numel() / 2**20, 1),
            "what": "static steps + single-layer mean correction from this draw, on the device"}


def time_decode(torch, ssdi8, cfg, inp, sc, K, W):
    """One decode token for every (batch, head) of the workload (ssdi8_decode_step): one replay
    of a graph of K chained steps after W warmup steps, bracketed by HIP events on the launch
    stream; the int8 state stays in HBM.
    Algorithmic bytes: the int8 state read and written, x and y, dt, the token's B_q and C_q."""
    import numpy as np
    Bt, H, P, G, N = cfg.batch, cfg.nheads, cfg.headdim, cfg.ngroups, cfg.dstate
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    f32 = lambda a: dev(np.asarray(a, np.float32))
    x = dev(inp["x"][:, 0])
    dt = f32(inp["dt_raw"][:, 0])
    aB, aC, aXs, aS, aCB = (f32(sc[k]) for k in ("alpha_B", "alpha_C", "alpha_Xs", "alpha_S",
                                                 "alpha_CB"))
    Bq = ssdi8.quantize_act(dev(inp["B"][:, :1]), "group", aB)[0].reshape(Bt, G, N)
    Cq = ssdi8.quantize_act(dev(inp["C"][:, :1]), "group", aC)[0].reshape(Bt, G, N)
    A, D, corr = f32(inp["A"]), f32(inp["D"]), f32(sc["corr"])
    state = torch.zeros((Bt, H, P, N), dtype=torch.int8, device="cuda")
    y = torch.empty_like(x)
    run = lambda: ssdi8.decode_step(x, dt, A, Bq, Cq, aB, aC, aXs, aS, aCB, state, D=D,
                                    corr=corr, y=y)
    for _ in range(W):
        run()
    torch.cuda.synchronize()
    # K chained steps captured in one HIP graph (per-launch host overhead excluded, as in a
    # captured serving loop); one replay is timed
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(K):
            run()
    graph.replay()
    ev = ssdi8.HipEvents(2)
    torch.cuda.synchronize()
    ev.record(0)
    graph.replay()
    ev.record(1)
    torch.cuda.synchronize()
    us = ev.elapsed_ms(0, 1) / K * 1e3
    ev.close()
    sx = 2 if cfg.dtype == "fp16" else 4
    nbytes = 2 * Bt * H * P * N + 2 * Bt * H * P * sx + 4 * Bt * H + 2 * Bt * G * N
    gbs = nbytes / (us * 1e-6) / 1e9
    return {"us": round(us, 2), "tokens_per_s": round(Bt / (us * 1e-6), 1),
            "algorithmic_bytes": nbytes, "GBps": round(gbs, 1),
            "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
            "what": f"one decode token of {Bt} sequences x {H} heads (int8 state in place)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="long-64k",
                    help="one of the synthetic layers; the default is the largest one-GPU "
                         "workload (65536 tokens x 80 heads)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--settle-s", type=float, default=0.3,
                    help="untimed steps after the warmup until the GPU has run the layer this "
                         "long (its clocks reach steady state under sustained load)")
    ap.add_argument("--eager", action="store_true",
                    help="time eager launches instead of replays of one captured HIP graph")
    ap.add_argument("--path", choices=("auto", "separate", "single"), default="auto",
                    help="separate ChunkState / StatePassing / ChunkScan kernels, the single "
                         "pass, or the library's automatic choice")
    ap.add_argument("--separate-quant", action="store_true",
                    help="quantize B and C with ssdi8_quantize_act before the chunk scan (three "
                         "calls) instead of handing them to ChunkBMM unquantized")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="after the timed region, run one plain device-to-device copy of this "
                         "many MiB (a known-size reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported by this build "
              "(the SSD path shards over batch/heads with no exchange; see DESIGN.md).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_21952_amd import ssdi8, synth

    cfg = synth.CONFIGS[args.workload]
    calib = os.path.join(ROOT, "tests", "golden", "calib", cfg.name + ".npz")
    with np.load(calib, allow_pickle=False) as z:
        sc = {k: z[k] for k in z.files}
    print(f"[bench] workload {cfg.name}: B={cfg.batch} L={cfg.seqlen} H={cfg.nheads} "
          f"P={cfg.headdim} N={cfg.dstate} G={cfg.ngroups} Q={cfg.chunk} {cfg.dtype}",
          file=sys.stderr, flush=True)
    inp = synth.draw(cfg, 1)
    torch.cuda.set_device(0)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    f32 = lambda a: dev(np.asarray(a, np.float32))
    x, dt, Bf, Cf = dev(inp["x"]), dev(inp["dt_raw"]), dev(inp["B"]), dev(inp["C"])
    A, D, corr = f32(inp["A"]), f32(inp["D"]), f32(sc["corr"])
    aB, aC, aXs, aS, aCB = (f32(sc[k]) for k in ("alpha_B", "alpha_C", "alpha_Xs", "alpha_S",
                                                 "alpha_CB"))
    Bq = torch.empty(Bf.shape, dtype=torch.int8, device="cuda")
    Cq = torch.empty(Cf.shape, dtype=torch.int8, device="cuda")
    y = torch.empty_like(x)
    ws = torch.empty(ssdi8.workspace_size(ssdi8.dims(cfg.batch, cfg.seqlen, cfg.nheads,
                                                     cfg.ngroups)), dtype=torch.uint8,
                     device="cuda")
    K, W = args.steps, args.warmup
    ev = ssdi8.HipEvents(7 * max(K, 1))

    def step(k=None, events=None):
        events = ev if events is None else events
        if args.separate_quant:
            # ssdi8_quantize_act for B and C, then the chunk scan on B_q, C_q
            if k is not None:
                events.record(7 * k)
            ssdi8.quantize_act(Bf, "group", aB, out=Bq)
            if k is not None:
                events.record(7 * k + 1)
            ssdi8.quantize_act(Cf, "group", aC, out=Cq)
            ssdi8.ssd_chunk_scan(x, dt, A, Bq, Cq, aB, aC, aXs, aS, aCB, D=D, corr=corr,
                                 workspace=ws, y=y, final_state=True, path=args.path,
                                 stage_events=None if k is None else events.group(7 * k + 2))
        else:
            # B and C handed over unquantized: ChunkBMM quantizes them with the static steps
            if k is not None:
                events.record(7 * k)
                events.record(7 * k + 1)
            ssdi8.ssd_chunk_scan(x, dt, A, None, None, aB, aC, aXs, aS, aCB, D=D, corr=corr,
                                 workspace=ws, y=y, final_state=True, path=args.path,
                                 B=Bf, C=Cf,
                                 stage_events=None if k is None else events.group(7 * k + 2))

    for _ in range(W):
        step()
    torch.cuda.synchronize()
    graph = None
    if not args.eager:
        # one step captured as a HIP graph on a side stream; the timed region replays it K times
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        for _ in range(W):
            graph.replay()
        torch.cuda.synchronize()
    # Settle: untimed steps until the GPU has run the layer for args.settle_s seconds.  Under
    # sustained load its clocks take tens of ms to reach steady state (2.7B-shaped layer, 10
    # steps per sample: 0.148, 0.165, 0.169, 0.164, 0.161, ... 0.141 ms per step by the 250th).
    settle_end = time.perf_counter() + args.settle_s
    settle_steps = 0
    while time.perf_counter() < settle_end:
        for _ in range(10):
            if graph is not None:
                graph.replay()
            else:
                step()
        settle_steps += 10
        torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for k in range(K):
        if graph is not None:
            graph.replay()
        else:
            step(k)
    t1.record()
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    ms_step = total_ms / K
    # the median over K more steps, each bracketed by its own events (an event between steps
    # adds a little, so the mean above comes from the uninterrupted run)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    marks[0].record()
    for k in range(K):
        if graph is not None:
            graph.replay()
        else:
            step()
        marks[k + 1].record()
    torch.cuda.synchronize()
    per_step = sorted(marks[k].elapsed_time(marks[k + 1]) for k in range(K))
    ms_median = per_step[K // 2] if K % 2 else 0.5 * (per_step[K // 2 - 1] + per_step[K // 2])
    if graph is not None:
        # per-kernel durations: K eager steps right after, with the library's stage events
        # (ChunkBMM and the scan kernel set theirs from their own dispatch: start and end)
        keep_busy(graph, ms_step)
        for k in range(K):
            step(k)
        torch.cuda.synchronize()
    # per-module averages over the timed steps (events on the launch stream)
    single = ssdi8.uses_single_pass(ssdi8.dims(cfg.batch, cfg.seqlen, cfg.nheads, cfg.ngroups),
                                    x.dtype, args.path)
    mods = SINGLE if single else MODULES
    names = (("quantize_B", "quantize_C") if args.separate_quant else ()) + mods
    per = {n: 0.0 for n in names}
    for k in range(K):
        base = 7 * k
        if args.separate_quant:
            per["quantize_B"] += ev.elapsed_ms(base, base + 1)
            per["quantize_C"] += ev.elapsed_ms(base + 1, base + 2)
        if single:
            # stage events 0-1: ChunkBMM's start and end; 3-4: the single pass's
            per["chunk_bmm"] += ev.elapsed_ms(base + 2, base + 3)
            per["single_pass"] += ev.elapsed_ms(base + 5, base + 6)
        else:
            for i, n in enumerate(MODULES):
                per[n] += ev.elapsed_ms(base + 2 + i, base + 3 + i)
    per = {n: v / K for n, v in per.items()}
    ev.close()
    abytes = algorithmic_bytes(cfg, quant_in_bmm=not args.separate_quant)
    stages = {n: {"us": round(per[n] * 1e3, 2),
                  "GBps": round(abytes[n] / (per[n] * 1e-3) / 1e9, 1),
                  "hbm_frac": round(abytes[n] / (per[n] * 1e-3) / 1e9 / HBM_PEAK_GBS, 3)}
              for n in names}
    # MFMA utilisation of the contraction kernels (these shapes sit far below the machine
    # balance, so the HBM fraction is the binding one; reported for completeness)
    for n, (i8, f16) in algorithmic_ops(cfg).items():
        if n not in per:
            continue
        sec = per[n] * 1e-3
        stages[n]["int8_tops"] = round(i8 / sec / 1e12, 1)
        stages[n]["int8_mfma_frac"] = round(i8 / sec / 1e12 / INT8_PEAK_TOPS, 4)
        if f16:
            stages[n]["fp16_tflops"] = round(f16 / sec / 1e12, 1)
            stages[n]["fp16_mfma_frac"] = round(f16 / sec / 1e12 / FP16_PEAK_TFLOPS, 4)
    dom = "single_pass" if single else "chunk_scan"
    # the single pass runs every step of the layer after ChunkBMM: its roofline takes the layer's
    # minimum bytes (B and C at the input width); the separate path's ChunkScan its own minimum
    rbytes = layer_min_bytes(cfg) if single else abytes[dom]
    ach = rbytes / (per[dom] * 1e-3) / 1e9
    tokens = cfg.batch * cfg.seqlen
    value = tokens / (ms_step * 1e-3)
    traffic = measured_traffic(dom, cfg.name)
    result = {
        "metric": "INT8 SSD chunk-scan tokens/s per layer",
        "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": ms_step, "ms_per_step_median": ms_median,
        "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int8+fp16", "data": "synthetic",
        "config": {"workload": cfg.name, "batch": cfg.batch, "seqlen": cfg.seqlen,
                   "nheads": cfg.nheads, "headdim": cfg.headdim, "dstate": cfg.dstate,
                   "ngroups": cfg.ngroups, "chunk": cfg.chunk, "io_dtype": cfg.dtype},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(ach, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes": rbytes,
                     "basis": ("layer minimum: x in, y out, dt, B and C at the input width, "
                               "final state" if single else
                               "ChunkScan minimum: x in, y out, dt, C_q, CB_q, P_in"),
                     "kernel_min_bytes": abytes[dom],
                     "overhead_bytes": single_pass_overhead(cfg) if single else {},
                     "avg_us": round(per[dom] * 1e3, 2)},
        "timing": ("K replays of one captured HIP graph; per-kernel times from K eager steps "
                   "queued behind ~50 ms of replays, from the library's stage events (ChunkBMM "
                   "and the scan kernel: their own dispatch start and end)"
                   if graph is not None else "eager launches"),
        "settle": {"seconds": args.settle_s, "steps": settle_steps,
                   "what": "untimed steps after the warmup, until the GPU has run the layer "
                           "this long (clocks at steady state)"},
        "layer_hbm_frac": round(layer_min_bytes(cfg) / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "path": ("single pass: ChunkBMM, then ChunkState + StatePassing + ChunkScan in one kernel"
                 if single else "separate ChunkBMM, ChunkState, StatePassing, ChunkScan kernels")
                + ("; B, C quantized by ssdi8_quantize_act first" if args.separate_quant
                   else "; B, C quantized inside ChunkBMM"),
        "stages": stages,
    }
    f16 = time_fp16(torch, ssdi8, cfg, x, dt, A, Bf, Cf, D, K, W)
    f16["int8_speedup"] = round(value / f16["tokens_per_s"], 3)
    result["fp16_baseline"] = f16
    result["decode"] = time_decode(torch, ssdi8, cfg, inp, sc, K, W)
    result["calibrate"] = time_calibrate(torch, ssdi8, cfg, x, dt, A, Bf, Cf, D, min(K, 5))
    # cold: every step after a 512 MiB scratch write that evicts the 256 MB Infinity Cache
    Kc = min(K, 20)
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cold_ms, cold_dom = [], []
    for k in range(Kc):
        scratch.fill_(k & 0xff)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        if graph is not None:
            graph.replay()
        else:
            step()
        c1.record()
        torch.cuda.synchronize()
        cold_ms.append(c0.elapsed_time(c1))
    ev2 = ssdi8.HipEvents(7 * Kc)
    for k in range(Kc):
        scratch.fill_(k & 0xff)
        step(k, events=ev2)
        torch.cuda.synchronize()
        # the dominant kernel (ChunkScan, or the single pass) runs between events 3 and 4
        cold_dom.append(ev2.elapsed_ms(7 * k + 5, 7 * k + 6))
    ev2.close()
    del scratch
    cms = sorted(cold_ms)[Kc // 2]
    cdom = sorted(cold_dom)[Kc // 2]
    result["cold"] = {
        "what": "median of %d steps, each after a 512 MiB scratch write (Infinity Cache evicted)"
                % Kc,
        "ms_per_step": round(cms, 4), "tokens_per_s": tokens / (cms * 1e-3),
        "dominant_kernel_us": round(cdom * 1e3, 2),
        "dominant_kernel_GBps": round(rbytes / (cdom * 1e-3) / 1e9, 1),
        "dominant_kernel_hbm_frac": round(rbytes / (cdom * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    peaks = measured_peaks(torch, ssdi8)
    result["measured_peaks"] = peaks
    result["roofline"]["frac_of_measured_copy"] = round(ach / peaks["hbm_copy_GBps"], 4)
    for n, st in stages.items():
        st["frac_of_measured_copy"] = round(st["GBps"] / peaks["hbm_copy_GBps"], 4)
        if "int8_tops" in st:
            st["int8_frac_of_measured"] = round(st["int8_tops"] / peaks["int8_mfma_TOPS"], 4)
    if args.copy_probe_mb > 0:
        n = args.copy_probe_mb << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample ...", file=sys.stderr,
              flush=True)
        cb = cpu_baseline(cfg, inp, sc, args.cpu_budget_s)
        cb["gpu_over_cpu"] = round(value / cb["value"], 1)
        result["cpu_baseline"] = cb
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
