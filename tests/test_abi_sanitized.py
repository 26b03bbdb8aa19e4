"""The C-ABI's host-side validation under AddressSanitizer and UBSan (no GPU).

tests/host_abi/abi_checks.cpp calls every entry point with each kind of invalid argument (and
once with valid ones, which reach the device check and return PG_EHIP without a GPU), linked
against the library's own source built with the sanitizers on its host code only
(-Xarch_host: device code is unchanged).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(600)
def test_abi_validation_is_clean_under_host_sanitizers(tmp_path):
    hipcc = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "abi_checks")
    san = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fno-sanitize-recover=undefined"]
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", *san,
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "paper_2506_05433_amd", "csrc", "pg_attn.hip"),
           os.path.join(ROOT, "tests", "host_abi", "abi_checks.cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               HIP_VISIBLE_DEVICES="")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = run.stdout + run.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert run.returncode == 0 and "OK (0 mismatches)" in run.stdout, out[-4000:]
