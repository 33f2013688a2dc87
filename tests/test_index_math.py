"""Host test of the clustering kernels' cell-index arithmetic (built from the
library's own header with hipcc as host code; no GPU needed)."""

import os
import shutil
import subprocess

import pytest

from paper_2512_07009_amd import build as libbuild

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="needs hipcc")
def test_cell_coord_clamped(tmp_path):
    exe = str(tmp_path / "index_math_test")
    r = subprocess.run([libbuild.hipcc(), "-std=c++17", "-O1", "-I", libbuild.CSRC,
                        os.path.join(HERE, "cpp", "index_math_test.cpp"), "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "index math ok" in r.stdout
