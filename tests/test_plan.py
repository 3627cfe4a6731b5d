"""CPU checks of the launch plans built by csrc/api.hip (no GPU needed): the
plan checker in plan_check.cpp is compiled with hipcc against the library's
host code and run over shapes x near-field distances x (B = I or not) x (one
stream / two streams)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.timeout(600)
def test_plan_coverage_order_and_races(tmp_path):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not os.path.exists(hipcc) and shutil.which("hipcc") is None:
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "plan_check")
    cmd = [hipcc, "-O2", "-std=c++17", "-w", "--offload-arch=gfx950",
           "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2608_06291_amd", "csrc"),
           "-o", exe, os.path.join(HERE, "plan_check.cpp")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=500)
    print(r.stdout[-2000:])
    assert r.returncode == 0, r.stdout[-4000:]
    assert "fails 0" in r.stdout
