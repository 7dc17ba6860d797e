"""Build libssdi8.so (HIP kernels + C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_2608_21952_amd.build          # or: from paper_2608_21952_amd.build import build

Every call recompiles.  Objects go to _build/ at the repository root; the shared library is
written next to this file (paper_2608_21952_amd/libssdi8.so) by an atomic rename.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build", "ssdi8")
LIB = os.path.join(PKG, "libssdi8.so")

ARCH = "gfx950"
SOURCES = ["api.hip", "quantize.hip", "chunk_bmm.hip", "chunk_state.hip", "state_pass.hip",
           "chunk_scan.hip", "decode.hip", "fp16_bmm.hip", "fp16_state.hip",
           "fp16_scan.hip", "calibrate.hip", "probe.hip"]

# -ffp-contract=off: no fused multiply-add where the arithmetic defines separate roundings.
# -packed-fp32-ops off: never emit packed fp32 arithmetic.
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
         "-Wall", "-Wno-unused-function", "-Xclang", "-target-feature", "-Xclang",
         "-packed-fp32-ops", f"-I{INCLUDE}", f"-I{CSRC}"]


# Per-source additions.  chunk_scan.hip: no wave-aggregated atomics, so that the single pass's
# ticket atomic returns in the background while the loads issued after it are in flight (the
# aggregated form reads its result, and waits for it, right away).
SOURCE_FLAGS = {"chunk_scan.hip": ["-mllvm", "-amdgpu-atomic-optimizer-strategy=None"]}


def flags_for(src: str) -> list:
    return [*FLAGS, *SOURCE_FLAGS.get(src, [])]


def hipcc() -> str:
    h = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    return h


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *flags_for(src), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(16, os.cpu_count() or 1)))
    with concurrent.futures.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
