"""Every HIP kernel compiles for gfx950 without private scratch memory or
vector-register spills.  The linear kernels are capped at 80 VGPRs (six waves per
SIMD, three blocks per CU); small code changes have pushed them over the cap,
where they spill to scratch and every decode pass slows down.  Compiles the
sources with the build's own flags and reads the compiler's resource
remarks (no GPU needed)."""
import os
import re
import subprocess

import pytest

from paper_2606_03113_amd import build as b

SOURCES = [s for s in b.SOURCES if s.endswith(".hip") and "__global__" in open(os.path.join(b.CSRC, s)).read()]


def _remarks(src, tmp_path):
    cmd = [b.HIPCC, "-x", "hip", *b.FLAGS, "--cuda-device-only", "-c", os.path.join(b.CSRC, src),
           "-o", str(tmp_path / (src + ".o")), "-Rpass-analysis=kernel-resource-usage"]
    p = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert p.returncode == 0, p.stderr[-2000:]
    kernels, cur = {}, None
    for line in p.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            kernels[cur] = {}
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+)", line)
        if cur and m:
            kernels[cur][m.group(1).strip()] = int(m.group(2))
    return kernels


@pytest.mark.skipif(not os.path.exists(b.HIPCC), reason="hipcc not installed")
@pytest.mark.parametrize("src", SOURCES)
def test_no_scratch_or_spills(src, tmp_path):
    kernels = _remarks(src, tmp_path)
    assert kernels, "no kernels reported for %s" % src
    # scalar spills go to vector-register lanes, not memory: not counted
    bad = {k: v for k, v in kernels.items() if v.get("ScratchSize", 0) or v.get("VGPRs Spill", 0)}
    assert not bad, bad


@pytest.mark.skipif(not os.path.exists(b.HIPCC), reason="hipcc not installed")
def test_linear_kernels_keep_three_blocks_per_cu(tmp_path):
    kernels = _remarks("linear.hip", tmp_path)
    capped = {k: v for k, v in kernels.items() if "8k_linearI" in k}
    assert capped
    for k, v in capped.items():
        assert v["VGPRs"] <= 80 and v["Occupancy"] >= 6, (k, v)
