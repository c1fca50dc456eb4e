"""The C ABI's host logic under AddressSanitizer + UndefinedBehaviorSanitizer.

Builds tests/abi_host_check.cpp together with the library sources (host code
instrumented, device code as usual) into a temporary directory and runs it:
argument validation, NULL handles, kernel-class name bounds, and a create
that fails in its first HIP call (no GPU in the CPU test environment), with
leak detection on.  Skipped where a GPU is visible (the failing create is the
point) or hipcc is missing.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1903_05133_amd", "csrc")
SOURCES = ["hieravg.hip", "k_data.hip", "k_gemm.hip", "k_delayed.hip", "k_head.hip", "k_avg.hip"]


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.skipif(_gpu_visible(), reason="checks the create failure path, which needs a machine without a GPU")
def test_host_abi_under_sanitizers(tmp_path):
    hipcc = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    if not shutil.which(hipcc):
        pytest.skip("hipcc not found")
    exe = str(tmp_path / "abi_host_check")
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "abi_host_check.cpp"), *[os.path.join(CSRC, s) for s in SOURCES],
           "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1", UBSAN_OPTIONS="halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
    print(run.stdout)
    assert run.returncode == 0, run.stdout + run.stderr[-4000:]
    assert "host checks ok" in run.stdout
