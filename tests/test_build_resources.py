"""Register and LDS budgets of the hot kernels, from the compiler's resource-usage remarks
(gfx950, the library's own flags): no VGPR spills and no scratch memory at all (a value
reloaded from scratch is a vector-memory load, which waits behind every load in flight), and
the single pass and the separate ChunkScan within four workgroups per CU (at most 128 VGPRs,
40 KB of LDS).  A few SGPRs may spill into the lanes of a VGPR (v_writelane / v_readlane, no
memory access): the single pass's instantiations with fp16 output hold 4-6 that way, counted in
their VGPRs."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2608_21952_amd import build as libbuild

CSRC = libbuild.CSRC


def _resources(src):
    cmd = [libbuild.hipcc(), *libbuild.flags_for(src), "-S", "--cuda-device-only", "-o",
           os.devnull, "-Rpass-analysis=kernel-resource-usage", os.path.join(CSRC, src)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    out, cur = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            cur = out.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[bytes/(?:block|lane)\])?: (\d+)", line)
        if m and cur is not None:
            cur[m.group(1).strip()] = int(m.group(2))
    return out


pytestmark = pytest.mark.skipif(shutil.which(libbuild.hipcc()) is None and
                                not os.path.exists(libbuild.hipcc()), reason="hipcc missing")


@pytest.mark.parametrize("src", ["chunk_scan.hip", "chunk_bmm.hip", "chunk_state.hip",
                                 "state_pass.hip", "quantize.hip", "decode.hip"])
def test_no_register_spills(src):
    res = _resources(src)
    assert res, f"no kernels found in {src}"
    for name, r in res.items():
        assert r.get("VGPRs Spill", 0) == 0, f"{name}: {r}"
        assert r["ScratchSize"] == 0, f"{name}: {r}"
        assert r.get("SGPRs Spill", 0) <= 8, f"{name}: {r}"


def test_chunk_scan_fits_four_workgroups_per_cu():
    for name, r in _resources("chunk_scan.hip").items():
        assert r["VGPRs"] + r.get("AGPRs", 0) <= 128, f"{name}: {r}"
        assert r["LDS Size"] <= 40 * 1024, f"{name}: {r}"
