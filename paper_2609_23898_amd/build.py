"""Compiles libcerar.so in-tree with hipcc for gfx950."""

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libcerar.so")
EXAMPLE_SRC = os.path.join(ROOT, "tests", "c_abi", "allreduce.c")
EXAMPLE = os.path.join(ROOT, "tests", "c_abi", "allreduce")

HIP_SOURCES = ["kernels.hip", "synth.hip"]
CXX_SOURCES = ["plan.cpp", "linalg.cpp"]

# Packed fp32 instructions stay disabled in every HIP translation unit.
HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wall", "-Wno-unused-result"]
CXX_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("command failed: " + " ".join(cmd))
    return r


def build(verbose=False):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    tmp = os.path.join(HERE, "_build")
    os.makedirs(tmp, exist_ok=True)
    objs = []
    for src in CXX_SOURCES:
        obj = os.path.join(tmp, src + ".o")
        _run(["g++", *CXX_FLAGS, "-I", os.path.join(ROOT, "include"), "-c",
              os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    for src in HIP_SOURCES:
        obj = os.path.join(tmp, src + ".o")
        _run([hipcc, *HIP_FLAGS, "-I", os.path.join(ROOT, "include"), "-c",
              os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    tmp_out = OUT + ".tmp"
    _run([hipcc, "-shared", "--offload-arch=gfx950", "-fPIC", *objs, "-o", tmp_out, "-lpthread"])
    os.replace(tmp_out, OUT)
    # a C consumer of the ABI alone (no Python), run by the GPU tests
    _run(["gcc", "-std=c11", "-O2", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
          "-I", "/opt/rocm/include", EXAMPLE_SRC, "-o", EXAMPLE, "-L", HERE, "-lcerar",
          "-L", "/opt/rocm/lib", "-lamdhip64", "-lm", "-Wl,-rpath,$ORIGIN/../../paper_2609_23898_amd", "-Wl,-rpath,/opt/rocm/lib"])
    if verbose:
        print("built", OUT, "and", EXAMPLE)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
