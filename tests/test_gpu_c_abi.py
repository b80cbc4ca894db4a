"""The C ABI on its own: tests/c_abi/allreduce.c (built by build()) runs one
all-reduce per plan through cerar.h and the HIP runtime, with no Python in
the process, and checks the result on the host (see its header)."""

import os
import subprocess

import pytest

from conftest import ROOT

pytestmark = pytest.mark.gpu

EXE = os.path.join(ROOT, "tests", "c_abi", "allreduce")


def test_c_program_uses_the_abi_alone():
    assert os.path.exists(EXE), "build() compiles tests/c_abi/allreduce"
    run = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(run.stdout)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "c-abi example ok" in run.stdout
