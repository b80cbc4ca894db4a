"""Host logic of bench.py, on the CPU: the algorithmic byte count of a step,
the launch families, the rocprofv3 summaries (on small synthetic CSV files
in rocprofv3's column layout) and the refusal of more than one GPU."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
from conftest import ROOT
from paper_2609_23898_amd import cerar as C


@pytest.mark.parametrize("N,c", [(2, 2), (2, 5), (4, 4), (4, 9), (8, 16), (8, 64), (16, 128), (64, 128)])
def test_step_bytes_match_the_stream_count(N, c):
    """Encode: c chunks read, c written, plus the message-1 copy.  Rounds
    1..N-1: receive + delta read, message written (3 streams); rounds N..c-1:
    receive, two deltas read, message written (4); rounds c..L-1: receive and
    one delta read, message written (3); round L only relabels.  Decode: L+1
    observations read, c outputs written.  Summed: (8c + 3N - 9) p floats."""
    p = 96
    b = C.phase_bytes_per_worker(N, c, p)
    L = c + N - 2
    assert sorted(b["rounds"]) == list(range(1, L + 1))
    assert b["rounds"][L] == 0
    total = b["encode"] + sum(b["rounds"].values()) + b["decode"]
    assert total == (8 * c + 3 * N - 9) * p * 4


def test_headline_step_bytes_and_launch_families():
    """N=8, c=64, d=1,414,647,808: p = 22,103,872 and 372,759,697,408 bytes
    per step; 7 rounds of K2, 56 of K3 with two deltas, 6 with one."""
    N, c, d = 8, 64, 1_414_647_808
    p = -(-d // c)
    assert p == 22_103_872 and p % 32 == 0
    b = C.phase_bytes_per_worker(N, c, p)
    assert N * (b["encode"] + sum(b["rounds"].values()) + b["decode"]) == 372_759_697_408
    L = c + N - 2
    fams = [bench.family_of(k, N, c, L) for k in range(1, L + 1)]
    assert fams.count("k_round<0> (K2: recv + delta)") == N - 1 == 7
    assert fams.count("k_round<1> (K3: recv - delta + delta)") == c - N == 56
    assert fams.count("k_round<2> (K3: recv - delta)") == N - 2 == 6
    assert fams[-1] is None
    per_launch = bench._launch_bytes()
    assert per_launch["k_round<1> (K3: recv - delta + delta)"] == N * 4 * p * 4
    assert per_launch["k_encode (K1)"] == N * (2 * c + 1) * p * 4


def test_kernel_names_map_to_families():
    assert bench.family_of_name("k_encode_dbuf<16, 4>") == "k_encode (K1)"
    assert bench.family_of_name("k_round<1, true>") == "k_round<1> (K3: recv - delta + delta)"
    assert bench.family_of_name("k_round<0, false>") == "k_round<0> (K2: recv + delta)"
    assert bench.family_of_name("k_decode_wide<48, 8>") == "k_decode (K4)"
    assert bench.family_of_name("k_encode_split<8>") == "k_encode (K1)"
    assert bench.family_of_name("k_decode_split<8>") == "k_decode (K4)"
    assert bench.family_of_name("k_copy4") == "k_copy4 (copy reference)"
    assert bench.family_of_name("k_fused_lanes<4, 8, true>") is None
    assert bench.family_of_name("k_norms") is None


def _write_csv(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as f:
        f.write(",".join(header) + "\n")
        for r in rows:
            f.write(",".join(str(x) for x in r) + "\n")


def test_counter_summary_is_scaled_by_the_copy_kernel(tmp_path):
    """FETCH_SIZE reads half the copy kernel's bytes (as on gfx950) and
    WRITE_SIZE all of them: both are divided by their copy-kernel factor."""
    copy_floats = 1 << 20
    copy_kib = copy_floats * 4 / 1024
    enc = "void cerar::(anonymous namespace)::k_encode_dbuf<16, 4>(cerar::(anonymous namespace)::EncParams)"
    hdr = ["Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"]
    g = copy_floats // 4
    # the bench's other copies (gradient refills, 3x as long) must not enter the scale
    _write_csv(str(tmp_path / "fetch" / "host" / "pmc_counter_collection.csv"), hdr,
               [["k_copy4", g, "FETCH_SIZE", copy_kib * 0.5], ["k_copy4", 3 * g, "FETCH_SIZE", copy_kib * 1.5],
                [f'"{enc}"', 4096, "FETCH_SIZE", 1000.0], [f'"{enc}"', 4096, "FETCH_SIZE", 1200.0]])
    _write_csv(str(tmp_path / "write" / "host" / "pmc_counter_collection.csv"), hdr,
               [["k_copy4", g, "WRITE_SIZE", copy_kib], ["k_copy4", 3 * g, "WRITE_SIZE", 3 * copy_kib],
                [f'"{enc}"', 4096, "WRITE_SIZE", 3000.0], [f'"{enc}"', 4096, "WRITE_SIZE", 3000.0]])
    out = tmp_path / "summary.txt"
    bench.summarize_pmc(str(tmp_path / "fetch"), str(tmp_path / "write"), str(out), copy_floats=copy_floats)
    text = out.read_text()
    assert "fetch_scale: 0.50000" in text and "write_scale: 1.00000" in text
    expect = (1100.0 / 0.5 + 3000.0) * 1024
    assert f"traffic_bytes_per_launch[k_encode (K1)]: {expect:.0f}" in text
    assert f"kernel_source_sha256: {bench.kernel_source_hash()}" in text


def test_trace_summary_compares_trace_and_event_averages(tmp_path):
    hdr = ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage"]
    _write_csv(str(tmp_path / "trace" / "host" / "trace_kernel_stats.csv"), hdr, [
        ['"void cerar::(anonymous namespace)::k_round<1, true>(cerar::(anonymous namespace)::RoundParams)"',
         10, 4_400_000, 440_000, 60.0],
        ['"void cerar::(anonymous namespace)::k_round<1, false>(cerar::(anonymous namespace)::RoundParams)"',
         10, 4_600_000, 460_000, 30.0],
        ['"void at::native::elementwise_kernel<128, 4>(int)"', 5, 500_000, 100_000, 10.0]])
    line = {"ms_per_step": 65.0, "value": 5700.0,
            "config": {"pct_hbm_peak": 71.3, "workload_name": "gpt2-small", "workload": "GPT-2-small N=8 c=32",
                       "plan": "kappa_max=1e3"},
            "roofline": {"kernel": "k_round<1> (K3: recv - delta + delta)", "achieved": 6300.0},
            "kernels": {"k_round<1> (K3: recv - delta + delta)": {"avg_ms": 0.459}}}
    log = tmp_path / "bench.log"
    log.write_text("some text\n" + json.dumps(line) + "\n")
    out = tmp_path / "trace.txt"
    bench.summarize_trace(str(tmp_path / "trace"), str(log), str(out),
                          bench_args=["--workload", "gpt2-small", "--cpu-positions", "0"])
    text = out.read_text()
    assert "on the gpt2-small workload" in text and "GPT-2-small N=8 c=32; plan: kappa_max=1e3" in text
    assert "-- python3 bench.py --workload gpt2-small --cpu-positions 0 > " in text
    rows = [r for r in text.splitlines() if r.startswith("k_round<1> (K3")]
    assert len(rows) == 1
    trace_avg, event_avg, ratio = (float(x) for x in rows[0].split()[-3:])
    assert trace_avg == pytest.approx(0.45) and event_avg == pytest.approx(0.459)
    assert ratio == pytest.approx(0.459 / 0.45, abs=1e-3)
    assert "other kernels (input generation, torch copies; untimed)" in out.read_text()


def test_more_than_one_gpu_is_refused():
    run = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=300)
    assert run.returncode == 2
    assert "--gpus 2 is not supported" in run.stderr
    assert run.stdout.strip() == ""


def test_committed_profiles_are_consistent():
    """The committed counter summary covers every timed family at the
    headline, its traffic per launch stays within 2 % below and 6 % above the
    algorithmic bytes (no re-reads), and the traced summaries agree with the
    bench's HIP events within 3 % for the launches that dominate the step."""
    import re as _re
    text = open(bench.TRAFFIC_FILE).read()
    algo = bench._launch_bytes()
    for fam, a in algo.items():
        m = _re.search(r"^traffic_bytes_per_launch\[" + _re.escape(fam) + r"\]: (\d+)", text, _re.M)
        assert m, fam
        assert 0.98 <= int(m.group(1)) / a <= 1.06, (fam, int(m.group(1)) / a)
    trace = open(os.path.join(ROOT, "profiles", "kernel_trace_cerar_n8_c64_pythia1.4b.txt")).read()
    for fam in ("k_encode (K1)", "k_decode (K4)", "k_round<1> (K3: recv - delta + delta)"):
        row = [r for r in trace.splitlines() if r.startswith(fam)]
        assert len(row) == 1, fam
        ratio = float(row[0].split()[-1])
        assert 0.97 <= ratio <= 1.03, (fam, ratio)
    for f in os.listdir(os.path.join(ROOT, "profiles")):
        assert f.endswith((".txt", ".md")), f
    # the c = 128 counter summary: the split-operand encode and decode and the
    # rounds move their algorithmic bytes
    path = bench.TRAFFIC_FILES["heavytail-n16-c128"]
    if os.path.exists(path):
        text = open(path).read()
        for fam, a in bench._launch_bytes("heavytail-n16-c128").items():
            m = _re.search(r"^traffic_bytes_per_launch\[" + _re.escape(fam) + r"\]: (\d+)", text, _re.M)
            assert m, fam
            assert 0.98 <= int(m.group(1)) / a <= 1.06, (fam, int(m.group(1)) / a)


def test_contraction_peak_names_the_split_kernels():
    """The c = 128 interior encode, and the decode with K <= 144, run six bf16
    MFMA products per fp32 product: their fp32-equivalent roof is the bf16
    peak over six, which puts their 32 flop per byte below the ridge (HBM
    bound); the other stages keep the fp32 MFMA peak."""
    peak, how = bench.contraction_peak("encode", 128, 143)
    assert abs(peak - 2500.0 / 6) < 1e-9 and "bf16" in how
    assert bench.contraction_peak("decode", 128, 144)[0] == peak
    assert bench.contraction_peak("decode", 128, 145)[0] == bench.FP32_MFMA_PEAK_TFLOPS
    assert bench.contraction_peak("encode", 64, 71)[0] == bench.FP32_MFMA_PEAK_TFLOPS
    assert 32 < peak * 1e12 / (bench.HBM_PEAK_GBS * 1e9)


def test_launch_bytes_use_the_library_chunk_length():
    """Per-launch algorithmic bytes of a workload whose d is not a multiple
    of 32 c: the chunk length is the library's (ceil(d / c) rounded up to 32)."""
    from paper_2609_23898_amd import synth
    wl = synth.workload("heavytail-n16-c128")
    plan = C.Plan.explicit(np.stack([np.eye(wl.c)] * wl.N), np.zeros((wl.N, wl.c + wl.N - 1, wl.c)))
    p, _ = plan.chunk_len(wl.d)
    assert p % 32 == 0 and p * wl.c >= wl.d and p != wl.d // wl.c
    b = bench._launch_bytes("heavytail-n16-c128")
    assert b["k_encode (K1)"] == wl.N * (2 * wl.c + 1) * p * 4
    assert b["k_decode (K4)"] == wl.N * (2 * wl.c + wl.N - 1) * p * 4
    assert b["k_round<1> (K3: recv - delta + delta)"] == wl.N * 4 * p * 4
