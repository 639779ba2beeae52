"""Register spills in the HIP kernels, from the compiler's resource-usage
remarks (hipcc for gfx950 on the CPU, no GPU needed).  A spill inside a tile
loop is costly here: the reload waits on vector memory, which completes in
issue order, so it also waits for every tile load in flight.  Every kernel
must compile without VGPR spills, except the rotary variants of the stream
decomposition, which spill a few values outside their tile loops."""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_02544_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Rotary stream variants: spills allowed up to this many VGPRs.
ALLOWED = {"attn_bf16_stream": 40}


def spills(source):
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-c",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Rpass-analysis=kernel-resource-usage",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(CSRC, source), "-o", os.devnull]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    out, name = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"VGPRs Spill: (\d+)", line)
        if m and name:
            out[name] = int(m.group(1))
    return out


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None,
                    reason="hipcc not available")
@pytest.mark.parametrize("source", ["simsd_attention.hip", "simsd_accept.hip", "simsd_lmhead.hip"])
def test_no_vgpr_spills(source):
    found = spills(source)
    assert found, "no kernel resource remarks parsed"
    bad = []
    for name, n in found.items():
        if n == 0:
            continue
        rotary_stream = "attn_bf16_stream" in name and re.search(r"ELb[01]ELb1EEEv", name)
        limit = ALLOWED["attn_bf16_stream"] if rotary_stream else 0
        if n > limit:
            bad.append((name, n))
    assert not bad, f"VGPR spills: {bad}"
