"""Every kernel of the library compiles for gfx950 without register spills
(no scratch memory per lane): a spilled accumulator or operand turns into
HBM traffic inside the hot loops.  Compiles each HIP source with the
compiler's kernel resource report (no GPU needed)."""

import os
import re
import shutil
import subprocess

import pytest

from paper_2512_07009_amd import build as libbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIP_SOURCES = [s for s in libbuild.SOURCES if s.endswith(".hip")]


def resource_report(src: str) -> list[dict]:
    out = os.path.join("/tmp", f"flock_ru_{os.getpid()}_{src}.o")
    cmd = [libbuild.hipcc(), "--offload-arch=" + libbuild.ARCH, "-O3", "-std=c++17", "-fPIC",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", libbuild.INCLUDE, "-I", libbuild.CSRC, "--cuda-device-only", "-c",
           os.path.join(libbuild.CSRC, src), "-o", out, "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if os.path.exists(out):
        os.remove(out)
    assert r.returncode == 0, r.stderr[-2000:]
    kernels, cur = [], None
    for line in r.stderr.splitlines():
        m = re.search(r"remark:\s+(Function Name|ScratchSize \[bytes/lane\]|VGPRs Spill|SGPRs Spill|VGPRs|AGPRs): (\S+)",
                      line)
        if not m:
            continue
        key, val = m.group(1), m.group(2)
        if key == "Function Name":
            cur = {"name": val}
            kernels.append(cur)
        elif cur is not None:
            cur[key] = val
    return kernels


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs hipcc")
@pytest.mark.parametrize("src", HIP_SOURCES)
def test_no_scratch_or_spills(src):
    kernels = resource_report(src)
    assert kernels, f"no kernels reported for {src}"
    bad = [(k["name"], k.get("ScratchSize [bytes/lane]"), k.get("VGPRs Spill"), k.get("SGPRs Spill"))
           for k in kernels
           if k.get("ScratchSize [bytes/lane]", "0") != "0" or k.get("VGPRs Spill", "0") != "0"]
    assert not bad, f"{src}: kernels with scratch or VGPR spills: {bad}"
