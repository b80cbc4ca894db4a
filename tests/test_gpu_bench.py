"""bench.py's one JSON line, on the smallest workload: the fields the
measurement contract asks for are present and consistent with each other
(value from the bytes and the step time, the roofline fraction from its
achieved and peak values, the CPU baseline from the oracle)."""

import json
import math
import os
import subprocess
import sys

import pytest

from conftest import ROOT

pytestmark = pytest.mark.gpu


def test_bench_line_on_the_tiny_workload():
    run = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny-n4-c4",
                          "--steps", "3", "--warmup", "1", "--cpu-positions", "256", "--cpu-seconds", "1", "--copy-floats", "65536"],
                         capture_output=True, text=True, timeout=300)
    assert run.returncode == 0, run.stderr[-3000:]
    lines = [l for l in run.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, run.stdout
    b = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in b, key
    assert b["n_gpus"] == 1 and b["steps"] == 3 and b["warmup"] == 1 and b["dtype"] == "f32"
    assert b["config"]["workload_name"] == "tiny-n4-c4" and "workload" in b["config"]
    assert abs(b["value"] - b["config"]["bytes_per_step"] / (b["ms_per_step"] * 1e-3) / 1e9) <= 0.01 * b["value"]
    r = b["roofline"]
    assert r["bound"] in ("hbm", "mfma") and r["peak"] > 0
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-3
    assert r["traffic"] is None                     # the counter summary covers the headline only
    cb = b["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0 and cb["sample"]
    assert 1 <= cb["threads"] <= min(cb["cores"], 15) and "GPU line's plan" in cb["plan"]
    ip = b["in_place_encode"]
    assert ip["ms_per_step_events"]["median"] > 0 and ip["encode_ms"]["median"] > 0
    sp = b["encode_spread"]
    assert 0 < sp["min_ms"] <= sp["max_ms"] and "fresh_buffer" in sp
    # the tiny workload's Vandermonde plan (tau = 0.5, Sec. II-B) is a poor
    # approximation by construction (Phi about 185), so only finiteness is checked
    assert math.isfinite(b["approx_rel_err_max"])
    assert b["plan_info"]["kappa_M"] > 0
