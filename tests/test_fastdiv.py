"""Host check of the multiply-high division the kernels use to decode workgroup indices.

The divisor constants are computed on the host (``FastDiv::make`` in the kernels' internal
header) and must reproduce exact unsigned division for every index below 2^31.  The check
compiles a small host program against that header and runs it; no GPU is involved.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2407_02109_amd", "csrc")


@pytest.mark.skipif(shutil.which("hipcc") is None, reason="hipcc not installed")
def test_fastdiv_exact(tmp_path):
    exe = str(tmp_path / "fastdiv_check")
    src = os.path.join(ROOT, "tests", "native", "fastdiv_check.cpp")
    subprocess.run(["hipcc", "-O2", "-std=c++17", "-I", CSRC, src, "-o", exe], check=True,
                   capture_output=True, timeout=300)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "fastdiv OK" in r.stdout
