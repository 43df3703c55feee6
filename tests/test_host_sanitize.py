"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

tests/host/abi_harness.cpp links the C ABI's host sources (validation,
planning, parameter set-up, the Mode A budget) against stub launchers that
check the launch parameters and launch nothing, and drives every entry point
with random valid descriptors and rejected ones.  The sanitizers apply to the
host code only (each -fsanitize flag is passed with -Xarch_host).  No GPU is
used.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_19868_amd", "csrc")


def _hipcc():
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return None


def test_abi_host_code_under_sanitizers(tmp_path):
    hipcc = _hipcc()
    if hipcc is None:
        pytest.skip("hipcc is not available")
    exe = str(tmp_path / "abi_harness")
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wno-unused-command-line-argument",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "api.hip"), os.path.join(CSRC, "mdm_plan.hip"),
           "-x", "hip", os.path.join(ROOT, "tests", "host", "abi_harness.cpp"), "-o", exe]
    b = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
    assert b.returncode == 0, b.stdout[-3000:]
    # the HIP runtime keeps its allocations to the end of the process: leaks are not checked
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout[-5000:]
    assert "Sanitizer" not in r.stdout and " 0 failures" in r.stdout, r.stdout[-3000:]
