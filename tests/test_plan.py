"""Work planning of the fused lm-head kernel, checked on the CPU.

tests/plan_check.cpp is compiled (host code only) against the same header
the library uses for its launch geometry and workspace layout, and sweeps
call sizes: every launch of a call must fit the workspace its plan sizes,
including calls whose hidden states exceed 4 GiB and are cut into a full
launch plus a smaller remainder, and every work item must be covered once.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_plan_arithmetic(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = tmp_path / "plan_check"
    src = os.path.join(ROOT, "tests", "plan_check.cpp")
    r = subprocess.run([hipcc, "-O2", "-std=c++17", "-x", "hip", "--offload-arch=gfx950", src, "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "plan_check: ok" in r.stdout
