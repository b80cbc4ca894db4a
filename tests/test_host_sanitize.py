"""The host plan builder (plan.cpp, linalg.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer: a g++ build of those files with a small driver,
no device code.  Skipped when g++ or the sanitizer runtimes are missing."""

import os
import shutil
import subprocess

import pytest

from conftest import ROOT

HERE = os.path.dirname(os.path.abspath(__file__))


def test_plan_builder_is_clean_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    csrc = os.path.join(ROOT, "paper_2609_23898_amd", "csrc")
    exe = str(tmp_path / "plan_driver")
    cmd = [gxx, "-std=c++17", "-g", "-O1", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", csrc,
           os.path.join(csrc, "plan.cpp"), os.path.join(csrc, "linalg.cpp"),
           os.path.join(HERE, "host_sanitize", "plan_driver.cpp"), "-o", exe, "-lpthread"]
    build = subprocess.run(cmd, capture_output=True, text=True)
    if build.returncode != 0 and "asan" in build.stderr.lower():
        pytest.skip("sanitizer runtime unavailable")
    assert build.returncode == 0, build.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "runtime error" not in run.stderr and "ERROR: AddressSanitizer" not in run.stderr
    assert "created 148" in run.stdout, run.stdout
