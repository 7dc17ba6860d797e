"""The exact in-chunk prefix sum the kernels fall back to when a chunk's decay increments span
too many binades for a tree of fp64 additions to be exact (ChunkCumsum, Alg. 2 module 1): the
same source (csrc/exact_sum.hpp), built for the host, against Python's correctly rounded
math.fsum, bit for bit."""
import math
import os
import shutil
import struct
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_21952_amd", "csrc")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("g++ missing")
    exe = str(tmp_path_factory.mktemp("exact_sum") / "drv")
    subprocess.run([cxx, "-O2", "-std=c++17", "-ffp-contract=off", f"-I{CSRC}",
                    os.path.join(ROOT, "tests", "exact_sum_driver.cpp"), "-o", exe], check=True)
    return exe


def _prefixes(exe, v):
    v = np.asarray(v, np.float32)
    r = subprocess.run([exe], input=struct.pack("<i", v.size) + v.tobytes(),
                       capture_output=True, check=True)
    return np.frombuffer(r.stdout, np.float64)


def _check(exe, v):
    v = np.asarray(v, np.float32)
    got = _prefixes(exe, v)
    ref = np.array([math.fsum(v[:i + 1].astype(np.float64)) for i in range(v.size)])
    assert got.view(np.uint64).tolist() == ref.view(np.uint64).tolist()


def _wide(rng, n, lo, hi, signs):
    e = rng.integers(lo, hi, n)
    m = rng.uniform(1.0, 2.0, n)
    s = rng.choice(signs, n)
    return (s * np.ldexp(m, e)).astype(np.float32)


def test_matches_fsum_on_wide_spans(driver):
    rng = np.random.default_rng(11)
    for _ in range(4):
        _check(driver, _wide(rng, 256, -149, 127, [-1.0]))       # one sign: decay increments
        _check(driver, _wide(rng, 256, -149, 127, [-1.0, 1.0]))  # both signs: cancellation
        _check(driver, _wide(rng, 256, -70, 8, [-1.0]))          # softplus over [-45, 25]


def test_matches_fsum_at_rounding_ties(driver):
    t = [1.0, 2.0 ** -53]                        # exactly half-way: ties to even (1.0)
    _check(driver, t)
    _check(driver, t + [2.0 ** -100])            # just above half-way: rounds up
    _check(driver, t + [-(2.0 ** -100)])         # just below: rounds down
    _check(driver, [1.0 + 2.0 ** -23, 2.0 ** -53, 2.0 ** -120, -(2.0 ** -140)])
    _check(driver, [-1.0, -(2.0 ** -53), -(2.0 ** -149)])


def test_matches_fsum_on_edge_values(driver):
    f32 = np.finfo(np.float32)
    tiny = np.float32(2.0 ** -149)
    _check(driver, [0.0, -0.0, tiny, -tiny, tiny, 0.0])
    _check(driver, [f32.max, f32.max, -f32.max, tiny, f32.max])
    _check(driver, [1.0] * 300 + [2.0 ** -60] * 5)
    _check(driver, [])
