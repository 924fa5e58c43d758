"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

``abi_sanitize_driver.cpp`` runs the library's planning, workspace sizing and
argument validation of every entry point (all without a kernel launch, so no
GPU is needed) with the library's source compiled in and the sanitizers on
the host side only (``-Xarch_host``); the device code is built as usual.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC) and shutil.which("hipcc") is None,
                    reason="needs hipcc")
def test_abi_host_code_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "abi_sanitize")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all"]
    cmd = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *san,
           "-I", os.path.join(ROOT, "include"), "-o", exe,
           os.path.join(HERE, "abi_sanitize_driver.cpp"),
           "-x", "hip", os.path.join(ROOT, "paper_2607_19456_amd", "csrc", "decode_attn.hip")]
    build = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert build.returncode == 0, build.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr[-2000:]
    assert "all checks passed" in run.stdout
