"""The fp64 log of the mutual-information kernel (csrc/fp64_log.h), built for the host with
hipcc and checked against the C library's log: at most one ulp apart (no GPU needed)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None,
                    reason="hipcc is not available")
def test_log_positive_within_one_ulp_of_libm(tmp_path):
    exe = str(tmp_path / "fp64_log_check")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O2", "-std=c++17",
           "-I", os.path.join(ROOT, "paper_2106_05373_amd", "csrc"),
           os.path.join(ROOT, "tests", "fp64_log_check.hip"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(run.stdout)
    assert run.returncode == 0, run.stdout + run.stderr
