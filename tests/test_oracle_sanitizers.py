"""The CPU oracle and the seeded input generator under AddressSanitizer and
UndefinedBehaviorSanitizer.

``oracle_sanitize_driver.c`` calls every oracle entry point (decode with and
without a head mask, the weights entry, single- and multi-row appends, the
multi-row decode) on small shapes covering the conventions' edge cases:
empty, negative and over-capacity lengths, d_k != d_v, MQA, T > 1, and the
shape errors.  Built with gcc (host code only; nothing here touches a GPU),
any invalid access or undefined operation aborts the run.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = [os.path.join(HERE, "oracle_sanitize_driver.c"),
           os.path.join(ROOT, "oracle", "oracle.c"),
           os.path.join(ROOT, "paper_2607_19456_amd", "csrc", "workload_rng.c")]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_sanitize")
    flags = ["-O1", "-g", "-std=c11", "-fopenmp", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    build = subprocess.run(["gcc", *flags, "-o", exe, *SOURCES, "-lm"],
                           capture_output=True, text=True)
    if build.returncode != 0 and "sanitizer" in build.stderr.lower():
        pytest.skip("gcc has no sanitizer runtime here: " + build.stderr[-200:])
    assert build.returncode == 0, build.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "all checks passed" in run.stdout
