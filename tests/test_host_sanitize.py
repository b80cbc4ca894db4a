"""The host plan builder (plan.cpp, linalg.cpp) in g++ builds with small
drivers, no device code:
  - under AddressSanitizer and UndefinedBehaviorSanitizer, every construction
    over a grid of (N, c) and the read-out calls;
  - with every allocation of a construction failing in turn: the C calls
    return CERAR_E_NOMEM or succeed, and leak nothing;
  - under ThreadSanitizer, plans built and one plan read from several threads
    at once, and the per-thread error text.
Skipped when g++ or a sanitizer runtime is missing."""

import os
import shutil
import subprocess

import pytest

from conftest import ROOT

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2609_23898_amd", "csrc")


def _build(tmp_path, driver, flags, runtime):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not found")
    exe = str(tmp_path / driver.replace(".cpp", ""))
    cmd = [gxx, "-std=c++17", "-g", "-O1", "-fno-omit-frame-pointer", *flags,
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "plan.cpp"), os.path.join(CSRC, "linalg.cpp"),
           os.path.join(HERE, "host_sanitize", driver), "-o", exe, "-lpthread"]
    build = subprocess.run(cmd, capture_output=True, text=True)
    if build.returncode != 0 and runtime in build.stderr.lower():
        pytest.skip(f"{runtime} runtime unavailable")
    assert build.returncode == 0, build.stderr[-2000:]
    return exe


def test_plan_builder_is_clean_under_sanitizers(tmp_path):
    exe = _build(tmp_path, "plan_driver.cpp", ["-fsanitize=address,undefined"], "asan")
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "runtime error" not in run.stderr and "ERROR: AddressSanitizer" not in run.stderr
    assert "created 148" in run.stdout, run.stdout


def test_plan_builder_survives_every_allocation_failure(tmp_path):
    exe = _build(tmp_path, "fault_driver.cpp", ["-fsanitize=undefined"], "ubsan")
    env = dict(os.environ, UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "runtime error" not in run.stderr
    last = run.stdout.strip().splitlines()[-1]
    assert last.startswith("fault points") and "bad 0, leaks 0" in last, last
    assert int(last.split("nomem ")[1].split(",")[0]) > 1000, last


def test_plan_builder_is_race_free_under_tsan(tmp_path):
    exe = _build(tmp_path, "thread_driver.cpp", ["-fsanitize=thread"], "tsan")
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    assert run.returncode == 0, (run.stdout + run.stderr)[-4000:]
    assert "ThreadSanitizer" not in run.stderr, run.stderr[-4000:]
    assert "threads done, failures 0" in run.stdout, run.stdout
