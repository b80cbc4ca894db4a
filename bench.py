#!/usr/bin/env python3
"""Throughput of the CERAR hot path on one MI355X.

One step = the whole approximate all-reduce for all N simulated workers:
encode (K1), rounds 1..L (K2/K3; round L only relabels) and decode (K4), on
synthetic gradients already resident in HBM.  The metric is the algorithmic
HBM traffic of the step, N * (8c + 3N - 9) * p * 4 bytes, divided by the
step time, in GB/s; its share of the 8 TB/s HBM peak is reported beside it.

Default workload: N = 8 workers, c = 64 chunks, d = 1,414,647,808 fp32
(Pythia-1.4B-shaped gradients with log-normal per-tensor scales), plan from
the condition-number-constrained design with kappa_max = 1e3.

The timed steps are single cerar_ring_simulate calls.  A second loop makes
the same launches through the per-step entry points with HIP events between
the phases on the launch stream; those events give each kernel's average
duration.  The fp64 CPU oracle is timed on sampled positions of the same
workload and plan (cpu_baseline), and the timed run's outputs are compared
with its results (parity_vs_oracle).
"""

import argparse
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "encode+round+decode GB/s per worker (% HBM peak), N=8 c=64 d=1.4e9 fp32"
HBM_PEAK_GBS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
BF16_MFMA_PEAK_TFLOPS = 2500.0
SPLIT_PRODUCTS = 6              # bf16 MFMA products per fp32 product in the split-operand kernels
CPU_WORKERS_MAX = 15
ORACLE_KEEP = 1024                 # oracle outputs kept per process for the GPU line's parity


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    from paper_2609_23898_amd import synth
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=synth.HEADLINE, choices=synth.WORKLOADS,
                    help="synthetic workload (default: the headline, pythia-1.4b)")
    ap.add_argument("--plan-iters", type=int, default=100, help="ALS iterations of the kappa design")
    ap.add_argument("--cpu-positions", type=int, default=1 << 14,
                    help="sampled positions per oracle process (0 = skip cpu_baseline)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="seconds each oracle process runs its sample (repeating it)")
    ap.add_argument("--copy-floats", type=int, default=1 << 30, help="size of the copy reference")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("TRACE_DIR", "BENCH_LOG", "OUT"),
                    help="write the summary of a rocprofv3 --kernel-trace --stats run of this bench")
    ap.add_argument("--traced-args", default="",
                    help="with --summarize-trace: the flags the traced bench.py run was given")
    ap.add_argument("--pmc-workload", default=None,
                    help="with --summarize-pmc: the workload the counter runs were taken on (default: the headline)")
    ap.add_argument("--summarize-pmc", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "OUT"),
                    help="write the HBM traffic summary of two rocprofv3 --pmc runs of this bench")
    return ap.parse_args()


# ---- rocprofv3 summaries ------------------------------------------------------

KERNEL_SOURCES = ("paper_2609_23898_amd/csrc/kernels.hip", "paper_2609_23898_amd/csrc/cerar_internal.hpp")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_cerar_n8_c64_pythia1.4b.txt")
# committed counter summaries per workload (the headline's is TRAFFIC_FILE)
TRAFFIC_FILES = {"pythia-1.4b": TRAFFIC_FILE,
                 "heavytail-n16-c128": os.path.join(ROOT, "profiles", "hbm_traffic_cerar_n16_c128_heavytail.txt")}
FAMILIES = (("k_encode", "k_encode (K1)"), ("k_round<0,", "k_round<0> (K2: recv + delta)"),
            ("k_round<1,", "k_round<1> (K3: recv - delta + delta)"),
            ("k_round<2,", "k_round<2> (K3: recv - delta)"), ("k_decode", "k_decode (K4)"),
            ("k_copy4", "k_copy4 (copy reference)"))


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def contraction_peak(stage, c, K):
    """Peak of a stage's contraction in fp32 TFLOP/s and how it runs.  At
    c = 128 the interior encode and the interior decode with K <= 144
    observations run on bf16 MFMAs with operands split into three bf16 terms,
    six products per fp32 product: their fp32-equivalent peak is the bf16 peak
    over six.  Every other encode and decode runs fp32 MFMAs."""
    if c == 128 and (stage == "encode" or K <= 144):
        return BF16_MFMA_PEAK_TFLOPS / SPLIT_PRODUCTS, "bf16 MFMA on three-term splits (6 products)"
    return FP32_MFMA_PEAK_TFLOPS, "fp32 MFMA"


def family_of_name(name):
    for key, fam in FAMILIES:
        if re.search(r"\b" + re.escape(key), name):
            return fam
    return None


def _find_csv(d, suffix):
    import glob
    hits = sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))
    if not hits:
        raise SystemExit(f"no *{suffix} under {d}")
    return hits[-1]


def _read_csv(path):
    import csv
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _launch_bytes(workload=None):
    """Algorithmic bytes per launch of each family at a workload (default: the
    Pythia-1.4B headline), with the library's chunk length: ceil(d / c)
    rounded up to a multiple of 32 floats."""
    from paper_2609_23898_amd import cerar as C
    from paper_2609_23898_amd import synth
    wl = synth.workload(workload or synth.HEADLINE)
    N, c = wl.N, wl.c
    p = -(-(-(-wl.d // c)) // 32) * 32
    bw = C.phase_bytes_per_worker(N, c, p)
    return {"k_encode (K1)": N * bw["encode"], "k_decode (K4)": N * bw["decode"],
            "k_round<0> (K2: recv + delta)": N * bw["rounds"][1],
            "k_round<1> (K3: recv - delta + delta)": N * bw["rounds"][N],
            "k_round<2> (K3: recv - delta)": N * bw["rounds"][c]}


def summarize_trace(trace_dir, bench_log, out_path, bench_args=()):
    """Summary of a rocprofv3 kernel trace of one bench.py run (bench_args:
    the flags that run was given, recorded in the command line)."""
    stats = _read_csv(_find_csv(trace_dir, "kernel_stats.csv"))
    bench = None
    with open(bench_log) as f:
        for line in f:
            if line.startswith("{"):
                bench = json.loads(line)
    rows, other = [], [0, 0.0, 0.0]
    for r in stats:
        if "cerar::" not in r["Name"] or "k_synth_fill" in r["Name"]:   # input generation, torch copies
            other[0] += int(r["Calls"])
            other[1] += float(r["TotalDurationNs"])
            other[2] += float(r["Percentage"])
            continue
        name = re.sub(r"^(void )?cerar::\(anonymous namespace\)::", "", r["Name"])
        name = re.sub(r"\(.*$", "", name)
        rows.append((name, int(r["Calls"]), float(r["TotalDurationNs"]), float(r["AverageNs"]),
                     float(r["Percentage"])))
    rows.sort(key=lambda x: -x[2])
    rows.append(("other kernels (input generation, torch copies; untimed)", other[0], other[1],
                 other[1] / max(other[0], 1), other[2]))
    cfg = bench["config"] if bench else {}
    name = cfg.get("workload_name", "pythia-1.4b")
    flags = " ".join(bench_args) if bench_args else ""
    lines = [f"# Kernel durations of bench.py on the {name} workload, rocprofv3 kernel trace",
             f"# workload: {cfg.get('workload', '?')}; plan: {cfg.get('plan', '?')}",
             "# command (repo root, MI355X):",
             f"#   rocprofv3 --kernel-trace --stats -f csv -d {trace_dir} -o trace -- python3 bench.py"
             f"{' ' + flags if flags else ''} > {bench_log}",
             f"#   python3 bench.py --summarize-trace {trace_dir} {bench_log} {out_path}",
             f"# kernel_source_sha256: {kernel_source_hash()}", "",
             f"{'kernel':<60s} {'calls':>6s} {'avg_us':>10s} {'total_ms':>10s} {'pct':>6s}"]
    fam_ns = {}
    for name, calls, tot, avg, pct in rows:
        short = name if len(name) <= 60 else name[:57] + "..."
        lines.append(f"{short:<60s} {calls:6d} {avg / 1e3:10.1f} {tot / 1e6:10.2f} {pct:6.2f}")
        # the bucketed call's batch kernels are listed but kept out of the
        # per-family comparison with the single-instance step's events
        fam = None if "_batch" in name else family_of_name(name)
        if fam:
            fam_ns.setdefault(fam, []).append((calls, tot))
    lines += ["", "# per family: trace average vs the bench's HIP-event average on the launch stream",
              f"{'family':<42s} {'trace_avg_ms':>12s} {'event_avg_ms':>12s} {'ratio':>7s}"]
    for fam, parts in fam_ns.items():
        ev = bench["kernels"].get(fam, {}).get("avg_ms") if bench else None
        if fam in ("k_encode (K1)", "k_decode (K4)") and len({n for n, _ in parts}) == 1:
            # one encode or decode is every listed kernel once (interior blocks,
            # then the masked tail), and the events bracket all of them
            ta = sum(t / n for n, t in parts) / 1e6
        else:                       # a round is one launch of one of the listed kernels
            ta = sum(t for _, t in parts) / sum(n for n, _ in parts) / 1e6
        lines.append(f"{fam:<42s} {ta:12.4f} {ev if ev is not None else float('nan'):12.4f} "
                     f"{(ev / ta) if ev else float('nan'):7.3f}")
    if bench:
        rf = bench["roofline"]
        lines += ["", f"# bench line: {bench['ms_per_step']} ms/step, {bench['value']} GB/s "
                      f"({bench['config']['pct_hbm_peak']}% of 8 TB/s); roofline kernel "
                      f"{rf['kernel']} at {rf['achieved']} {rf.get('unit', 'GB/s')} ({rf.get('bound', 'hbm')} bound)"]
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _pmc_per_family(d, counter, copy_grid=None):
    """Mean counter value per launch of each family, and the launch count.
    An encode or decode launch can be two dispatches (the interior blocks'
    kernel and the tail's), so a family's total is divided by its dispatches
    over its distinct kernel names.  The copy kernel also serves the bench's
    refills of other sizes: with copy_grid, only its dispatches of that grid
    size (the reference copy) count."""
    rows = _read_csv(_find_csv(d, "counter_collection.csv"))
    acc = {}
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        name = r["Kernel_Name"]
        fam = None if "_batch" in name else family_of_name(name)
        if fam is None:
            continue
        if fam.startswith("k_copy4") and copy_grid is not None and int(r["Grid_Size"]) != copy_grid:
            continue
        v, n, names = acc.get(fam, (0.0, 0, set()))
        acc[fam] = (v + float(r["Counter_Value"]), n + 1, names | {name})
    out = {}
    for fam, (v, n, names) in acc.items():
        launches = n // len(names)
        out[fam] = (v / launches, launches)
    return out


def summarize_pmc(fetch_dir, write_dir, out_path, copy_floats=1 << 30, workload=None):
    from paper_2609_23898_amd import synth
    fetch = _pmc_per_family(fetch_dir, "FETCH_SIZE", copy_grid=copy_floats // 4)
    write = _pmc_per_family(write_dir, "WRITE_SIZE", copy_grid=copy_floats // 4)
    copy = "k_copy4 (copy reference)"
    copy_kib = copy_floats * 4 / 1024.0
    f_scale = fetch[copy][0] / copy_kib
    w_scale = write[copy][0] / copy_kib
    algo = _launch_bytes(workload)
    wl = synth.workload(workload or synth.HEADLINE)
    wflag = f" --workload {workload}" if workload else ""
    lines = ["# HBM traffic per launch from rocprofv3 counters (FETCH_SIZE, WRITE_SIZE in KiB; an encode or "
             "decode launch is its interior and tail dispatches)",
             f"# workload: {wl.name} (N={wl.N}, c={wl.c}, d={wl.d}, fp32)",
             "# commands (repo root, MI355X), one counter per run:",
             "#   rocprofv3 --pmc FETCH_SIZE --kernel-include-regex 'k_(encode|round|decode|copy4)' -f csv "
             f"-d {fetch_dir} -o pmc -- python3 bench.py{wflag} --steps 1 --warmup 0 --cpu-positions 0",
             "#   rocprofv3 --pmc WRITE_SIZE --kernel-include-regex 'k_(encode|round|decode|copy4)' -f csv "
             f"-d {write_dir} -o pmc -- python3 bench.py{wflag} --steps 1 --warmup 0 --cpu-positions 0",
             f"#   python3 bench.py --summarize-pmc {fetch_dir} {write_dir} {out_path}"
             + (f" --pmc-workload {workload}" if workload else ""),
             "# scale: each counter divided by what it reads for the plain copy kernel k_copy4 moving "
             f"{copy_floats} floats ({copy_kib:.0f} KiB read and written per dispatch)",
             f"kernel_source_sha256: {kernel_source_hash()}",
             f"fetch_scale: {f_scale:.5f}", f"write_scale: {w_scale:.5f}", "",
             f"{'family':<42s} {'n':>4s} {'FETCH_KiB':>14s} {'WRITE_KiB':>14s} {'traffic_B':>16s} "
             f"{'algorithmic_B':>16s} {'ratio':>7s}"]
    for fam in [f for _, f in FAMILIES]:
        if fam not in fetch or fam not in write:
            continue
        fk, n = fetch[fam]
        wk, _ = write[fam]
        traffic = (fk / f_scale + wk / w_scale) * 1024.0
        a = algo.get(fam, 2 * copy_floats * 4)
        lines.append(f"{fam:<42s} {n:4d} {fk:14.1f} {wk:14.1f} {traffic:16.0f} {a:16d} {traffic / a:7.4f}")
        lines.append(f"traffic_bytes_per_launch[{fam}]: {traffic:.0f}")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def committed_traffic(family, workload=None):
    """HBM bytes per launch of `family` from the workload's committed counter
    summary, or None when there is none or the kernels changed since it was
    taken."""
    path = TRAFFIC_FILES.get(workload or "pythia-1.4b")
    if path is None:
        return None
    try:
        with open(path) as f:
            text = f.read()
    except OSError:
        return None
    m = re.search(r"^kernel_source_sha256: (\w+)", text, re.M)
    if not m or m.group(1) != kernel_source_hash():
        return None
    m = re.search(r"^traffic_bytes_per_launch\[" + re.escape(family) + r"\]: (\d+)", text, re.M)
    return int(m.group(1)) if m else None


def product_plan(C, wl, iters):
    if wl.N == 4 and wl.c == 4:
        return C.Plan(wl.N, wl.c, "vandermonde", 0.5), "Vandermonde tau=0.5 (Chebyshev nodes)"
    if wl.c == 16:
        return C.Plan(wl.N, wl.c, "o_eps", 1e-3, seed=1000 + wl.N), "O(eps) eps=1e-3"
    if wl.c == 128:
        return C.Plan(wl.N, wl.c, "o_eps", 1e-2, seed=1000 + wl.N), "O(eps) eps=1e-2"
    return (C.Plan(wl.N, wl.c, "kappa", 1e3, seed=1000 + wl.N, eps0=0.3, als_iters=iters, als_order=1),
            f"kappa_max=1e3 ALS {iters} it (projection before each R-step) from O(0.3)")


def family_of(k, N, c, L):
    if k <= N - 1:
        return "k_round<0> (K2: recv + delta)"
    if k < L:
        return "k_round<1> (K3: recv - delta + delta)" if k + 1 <= c else "k_round<2> (K3: recv - delta)"
    return None


def _oracle_worker(name, pos, U, R, seconds, keep, barrier, queue):
    """One host process of the CPU baseline: draws the oracle's inputs at its
    positions from the shared generator, waits for the other processes, then
    runs the fp64 oracle (encode, Algorithm 1 in lock-step, decode) on one
    thread, repeatedly until `seconds` have passed."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle import ring as OR
    from paper_2609_23898_amd import synth
    try:
        wl = synth.workload(name)
        N, c = wl.N, wl.c
        p = OR.chunk_len(wl.d, c, 32)               # the library's chunk length (cerar_chunk_len)
        flat = (np.arange(c)[None, :] * p + pos[:, None]).astype(np.int64)
        G = [wl.values_np(w, flat.ravel()).reshape(flat.shape).astype(np.float64) for w in range(N)]
        barrier.wait()
        reps, finite = 0, True
        with threadpool_limits(limits=1):
            t0 = time.time()
            while True:
                out = OR.allreduce_chunks(G, U, R)
                reps += 1
                t1 = time.time()
                if t1 - t0 >= seconds:
                    break
        finite = all(bool(np.all(np.isfinite(o))) for o in out)
        # the oracle's outputs at the first `keep` positions, for the GPU line's parity
        keep_pos = pos[:keep]
        keep_out = np.stack([o[:keep] for o in out])            # N x keep x c
        queue.put((t0, t1, reps * len(pos), finite, None, keep_pos, keep_out))
    except Exception as e:                          # reported by the parent
        try:
            barrier.abort()
        except Exception:
            pass
        queue.put((0.0, 0.0, 0, False, repr(e), None, None))


def cpu_baseline(name, U, R, plan_desc, positions, seconds):
    """Time the fp64 oracle on the GPU line's own plan (U, R from the
    library's plan) over sampled positions of the same workload: one worker
    process per host core available to this process, each single-threaded on its
    own positions.  Runs before the process touches the GPU, so the workers
    are plain forks of a process with no device state."""
    import multiprocessing as mp

    import numpy as np

    from oracle import ring as OR
    from paper_2609_23898_amd import synth

    wl = synth.workload(name)
    N, c, d = wl.N, wl.c, wl.d
    p = OR.chunk_len(d, c, 32)
    cores = os.cpu_count() or 1
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = cores
    # at most CPU_WORKERS_MAX workers, so that with the parent at most 16 processes run
    threads = max(1, min(usable, CPU_WORKERS_MAX))
    rng = np.random.default_rng(12345)
    per = max(1, min(positions, p // threads))
    pos_all = np.unique(np.concatenate([rng.integers(0, p, size=per * threads - 1), [p - 1]]))
    parts = np.array_split(pos_all, threads)
    ctx = mp.get_context("fork")
    barrier, queue = ctx.Barrier(threads), ctx.Queue()
    procs = [ctx.Process(target=_oracle_worker, args=(name, part, U, R, seconds, ORACLE_KEEP, barrier, queue))
             for part in parts]
    for pr in procs:
        pr.start()
    res = [queue.get(timeout=600) for _ in procs]
    for pr in procs:
        pr.join()
    errors = [r[4] for r in res if r[4]]
    if errors:
        raise RuntimeError(f"cpu_baseline worker failed: {errors[0]}")
    assert all(r[3] for r in res), "oracle output is not finite"
    per_pos = N * (8 * c + 3 * N - 9) * 4           # algorithmic bytes per position, all workers
    wall = max(r[1] for r in res) - min(r[0] for r in res)
    done = sum(r[2] for r in res)
    rates = sorted(r[2] * per_pos / (r[1] - r[0]) / 1e9 for r in res)
    step_bytes = N * (8 * c + 3 * N - 9) * p * 4
    value = done * per_pos / wall / 1e9
    reference = (np.concatenate([r[5] for r in res]), np.concatenate([r[6] for r in res], axis=1))
    return reference, {"value": round(value, 4), "unit": "GB/s", "cores": cores, "threads": threads, "kind": "oracle",
            "seconds": round(wall, 2), "per_thread_gbps_median": round(rates[len(rates) // 2], 4),
            "extrapolated_step_s": round(step_bytes / (value * 1e9), 1),
            "plan": "the GPU line's plan (its fp64 U and R, from cerar_plan_get_matrices)",
            "sample": f"{len(pos_all)} sampled positions x {c} chunks x {N} workers of the same workload, split "
                      f"over {threads} single-threaded processes (host: {cores} cores), each running the fp64 NumPy "
                      f"oracle (encode, Algorithm 1 lock-step, decode) on its positions repeatedly for "
                      f"{seconds:g} s ({done} positions in all); plan: {plan_desc}; GB/s counts the same "
                      f"algorithmic bytes per position as the GPU line"}


def _span_stats(xs):
    xs = sorted(xs)
    return {"median": round(xs[len(xs) // 2], 4), "min": round(xs[0], 4), "max": round(xs[-1], 4),
            "mean": round(sum(xs) / len(xs), 4)}


def in_place_steps(C, plan, d, grads, work, ws, out, steps):
    """Steps with work == grads: before each step the work rows are refilled
    with the gradients (and the zero pad) by the copy kernel; events bracket
    encode..decode only.  Returns the per-step spans and the encode times."""
    import torch
    N, c = plan.N, plan.c
    p, _ = plan.chunk_len(d)
    spans, enc = [], []
    for s in range(steps + 1):                     # the first step warms up
        for w in range(N):
            C.copy_f32(work[w, :d], grads[w])
        if c * p > d:
            work[:, d:c * p].zero_()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev[0].record()
        C.encode_round(plan, 0, d, work, work, ws)
        ev[1].record()
        for k in range(1, plan.L + 1):
            C.encode_round(plan, k, d, work, work, ws)
        C.decode(plan, d, work, ws, out)
        ev[2].record()
        torch.cuda.synchronize()
        if s > 0:
            spans.append(ev[0].elapsed_time(ev[2]))
            enc.append(ev[0].elapsed_time(ev[1]))
    return {"steps": steps, "ms_per_step_events": _span_stats(spans), "encode_ms": _span_stats(enc),
            "note": "work == grads (Sec. II storage rule); gradients restored by a copy before each step, "
                    "outside the events"}


def encode_spread(C, plan, d, grads, work, ws, reps):
    """The out-of-place encode timed on the bench's gradient buffer and on a
    second, freshly allocated copy of it (the encode's rate depends on the
    physical backing of the allocation it reads)."""
    import torch
    second = torch.empty_like(grads)
    for w in range(plan.N):
        C.copy_f32(second[w], grads[w])
    res = {}
    for name, g in (("bench_buffer", grads), ("fresh_buffer", second)):
        C.encode_round(plan, 0, d, g, work, ws)
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            C.encode_round(plan, 0, d, g, work, ws)
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        res[name] = _span_stats(ts)
    del second
    torch.cuda.empty_cache()
    allv = [res[k]["median"] for k in res]
    res["min_ms"], res["max_ms"] = min(allv), max(allv)
    return res


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace, bench_args=args.traced_args.split())
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, copy_floats=args.copy_floats, workload=args.pmc_workload)
        return
    if args.gpus != 1:
        print(f"bench.py runs the single-GPU simulation of all N workers; --gpus {args.gpus} is not "
              "supported (this implementation runs all workers on one GPU)", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2609_23898_amd import cerar as C
    from paper_2609_23898_amd import synth

    wl = synth.workload(args.workload)
    N, c, d = wl.N, wl.c, wl.d
    t = time.perf_counter()
    plan, plan_desc = product_plan(C, wl, args.plan_iters)          # host fp64, no device call
    info = plan.info()
    log(f"plan: {plan_desc} kappa_M={info['kappa_M']:.3g} phi={info['phi']:.4g} "
        f"({time.perf_counter() - t:.1f}s)")
    L = plan.L
    p, _ = plan.chunk_len(d)
    # the oracle on the host cores, before this process touches the GPU
    cpu = None
    if args.cpu_positions > 0:
        t = time.perf_counter()
        U_plan, R_plan = plan.matrices()
        oracle_ref, cpu = cpu_baseline(args.workload, U_plan, R_plan, plan_desc, args.cpu_positions,
                                       args.cpu_seconds)
        log(f"cpu baseline: {cpu['value']:.3f} GB/s on {cpu['threads']} processes "
            f"({time.perf_counter() - t:.1f}s total)")

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    dev = "cuda:0"

    t = time.perf_counter()
    grads = torch.empty((N, d), dtype=torch.float32, device=dev)
    for w in range(N):
        C.synth_fill(grads[w], wl, w)               # K6: the seeded generator on the device
    work, ws, out = C.allocate(plan, d, dev)
    torch.cuda.synchronize()
    log(f"inputs: N={N} c={c} d={d} p={p} L={L} generated in {time.perf_counter() - t:.1f}s; "
        f"{(grads.numel() + work.numel() + out.numel()) * 4 / 1e9 + ws.numel() / 1e9:.1f} GB resident")

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        C.encode_round(plan, 0, d, grads, work, ws)
        if ev is not None:
            ev[1].record()
        for k in range(1, L + 1):
            C.encode_round(plan, k, d, grads, work, ws)
            if ev is not None:
                ev[k + 1].record()
        C.decode(plan, d, work, ws, out)
        if ev is not None:
            ev[L + 2].record()

    for _ in range(args.warmup):
        C.ring_simulate(plan, d, grads, work, ws, out)
    torch.cuda.synchronize()
    # the timed steps: one cerar_ring_simulate call each (encode, rounds 1..L
    # and decode for all workers), with nothing else on the stream
    t0 = time.perf_counter()
    for _ in range(args.steps):
        C.ring_simulate(plan, d, grads, work, ws, out)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step")

    # per-kernel durations: the same launches through the per-step entry
    # points, with HIP events between the phases on the launch stream (each
    # event adds a few microseconds to the stream, so these steps are not the
    # timed ones)
    step()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(L + 3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for s in range(args.steps):
        step(events[s])
    torch.cuda.synchronize()
    ms_events = (time.perf_counter() - t2) * 1e3 / args.steps

    # the single-GPU fused variant (reported beside the ring, never as the value)
    fused = None
    if c % 16 == 0 and c <= 64 and (N <= 8 or c <= 32) and d % 4 == 0:
        C.ring_simulate_fused(plan, d, grads, out)
        torch.cuda.synchronize()
        t4 = time.perf_counter()
        for _ in range(args.steps):
            C.ring_simulate_fused(plan, d, grads, out)
        torch.cuda.synchronize()
        ms_f = (time.perf_counter() - t4) * 1e3 / args.steps
        step_bytes_ring = N * C.algorithmic_bytes_per_worker(N, c, p)
        fused = {"ms_per_step": round(ms_f, 4),
                 "ring_equivalent_gbps": round(step_bytes_ring / (ms_f * 1e-3) / 1e9, 1),
                 "moved_gbps": round(2 * N * d * 4 / (ms_f * 1e-3) / 1e9, 1),
                 "tflops": round(N * sum(C.phase_flops_per_worker(N, c, p).values()) / (ms_f * 1e-3) / 1e12, 1),
                 "note": "one kernel, all workers' messages on chip: only the gradients are read and the "
                         "outputs written; possible only when every worker shares one device, so it is "
                         "not the counted ring path"}
        log(f"fused single-GPU variant: {ms_f:.3f} ms/step")

    # workloads with DDP buckets: the bucketed call (one CERAR instance per bucket)
    bucketed = None
    if wl.buckets:
        lens = [b[1] for b in wl.buckets]
        wf, wsb = plan.bucketed_sizes(lens)
        bwork = torch.empty((N, wf), dtype=torch.float32, device=dev)
        bws = torch.empty(wsb, dtype=torch.uint8, device=dev)
        C.ring_simulate_bucketed(plan, wl.buckets, grads, bwork, bws, out)
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        for _ in range(args.steps):
            C.ring_simulate_bucketed(plan, wl.buckets, grads, bwork, bws, out)
        torch.cuda.synchronize()
        ms_b = (time.perf_counter() - t3) * 1e3 / args.steps
        bbytes = sum(N * C.algorithmic_bytes_per_worker(N, c, plan.chunk_len(ln)[0]) for ln in lens)
        bucketed = {"buckets": len(lens), "ms_per_step": round(ms_b, 4),
                    "gbps": round(bbytes / (ms_b * 1e-3) / 1e9, 1)}
        log(f"bucketed ({len(lens)} buckets): {ms_b:.3f} ms/step, {bucketed['gbps']} GB/s")
        del bwork, bws

    # per-kernel durations from the events
    fam_time, fam_count, fam_bytes = {}, {}, {}
    bw = C.phase_bytes_per_worker(N, c, p)
    flops = C.phase_flops_per_worker(N, c, p)

    def add(name, ms, nbytes):
        fam_time[name] = fam_time.get(name, 0.0) + ms
        fam_count[name] = fam_count.get(name, 0) + 1
        fam_bytes[name] = nbytes

    for ev in events:
        add("k_encode (K1)", ev[0].elapsed_time(ev[1]), N * bw["encode"])
        for k in range(1, L + 1):
            fam = family_of(k, N, c, L)
            if fam:
                add(fam, ev[k].elapsed_time(ev[k + 1]), N * bw["rounds"][k])
        add("k_decode (K4)", ev[L + 1].elapsed_time(ev[L + 2]), N * bw["decode"])
    kernels = {}
    for name in fam_time:
        avg = fam_time[name] / fam_count[name]
        kernels[name] = {"launches_per_step": fam_count[name] // args.steps,
                         "avg_ms": avg, "ms_per_step": fam_time[name] / args.steps,
                         "bytes_per_launch": fam_bytes[name],
                         "gbps": fam_bytes[name] / (avg * 1e-3) / 1e9}
    for name, key in (("k_encode (K1)", "encode"), ("k_decode (K4)", "decode")):
        peak, how = contraction_peak(key, c, L + 1)
        kernels[name]["tflops"] = N * flops[key] / (kernels[name]["avg_ms"] * 1e-3) / 1e12
        kernels[name]["contraction"] = how
        kernels[name]["mfma_peak_tflops"] = round(peak, 1)
        kernels[name]["mfma_frac"] = kernels[name]["tflops"] / peak
    for name in kernels:                            # every family against the HBM peak
        kernels[name]["hbm_frac"] = kernels[name]["gbps"] / HBM_PEAK_GBS
    # per-step spans (first event to last) of the timed loop: the paper reports
    # the median over runs (appendix, details of the numerical experiments);
    # the value above is the mean over the timed steps
    spans = sorted(ev[0].elapsed_time(ev[L + 2]) for ev in events)
    step_spans = {"median": round(spans[len(spans) // 2], 4), "min": round(spans[0], 4),
                  "max": round(spans[-1], 4)}
    dominant = max(kernels, key=lambda n: kernels[n]["ms_per_step"])
    dk = kernels[dominant]
    # the dominant kernel's roof: MFMA when its flops per algorithmic byte
    # exceed the ridge of its contraction's peak and the HBM peak, else HBM
    mfma_bound = "tflops" in dk and (
        dk["tflops"] * 1e12 / (dk["gbps"] * 1e9) > dk["mfma_peak_tflops"] * 1e12 / (HBM_PEAK_GBS * 1e9))
    if mfma_bound:
        roofline = {"bound": "mfma", "kernel": dominant, "achieved": round(dk["tflops"], 1),
                    "peak": dk["mfma_peak_tflops"], "unit": "TFLOP/s", "frac": round(dk["mfma_frac"], 4),
                    "traffic": None}
    else:
        roofline = {"bound": "hbm", "kernel": dominant, "achieved": round(dk["gbps"], 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(dk["gbps"] / HBM_PEAK_GBS, 4),
                    # from the workload's committed counter summary, where there is one
                    "traffic": committed_traffic(dominant, args.workload)}

    # achievable-bandwidth reference: a plain copy kernel
    nf = min(args.copy_floats, grads.numel())
    src = grads.view(-1)[:nf]
    dst = out.view(-1)[:nf]
    for _ in range(2):
        C.copy_f32(dst, src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        C.copy_f32(dst, src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbps = 2 * nf * 4 * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9

    # the paper's storage rule (Sec. II, initialisation: Delta_i overwrites G_i):
    # the same step with the encode in place, on the work buffer refilled from
    # the gradients before every step, outside the step's event span
    in_place = in_place_steps(C, plan, d, grads, work, ws, out, max(1, min(args.steps, 20)))
    log(f"in-place encode: {in_place['ms_per_step_events']['median']:.3f} ms/step (event spans), "
        f"encode {in_place['encode_ms']['median']:.3f} ms")
    # the encode's spread over gradient allocations: the same encode on a
    # second, freshly allocated copy of the gradients
    spread = encode_spread(C, plan, d, grads, work, ws, 10)
    log(f"encode on two gradient allocations: {spread}")

    # approximation error of the decoded sums (K5, not timed)
    C.ring_simulate(plan, d, grads, work, ws, out)
    norms = torch.empty(N + 1, dtype=torch.float64, device=dev)
    C.error_norms(N, d, grads, out, norms)
    nm = norms.cpu().numpy()
    rel_err = [math.sqrt(nm[i] / nm[N]) for i in range(N)]
    # parity of this run's outputs with the oracle at the CPU baseline's
    # positions (K5's parity term, cerar_sampled_norms)
    parity = None
    if cpu is not None:
        pos, ref = oracle_ref                                  # ref: N x S x c, chunk m at position e
        flat = (np.arange(c)[None, :] * p + pos[:, None])      # S x c flat output indices
        ok = flat < d
        idx = torch.from_numpy(np.ascontiguousarray(flat[ok], dtype=np.int64)).to(dev)
        refv = torch.from_numpy(np.ascontiguousarray(ref[:, ok])).to(dev)
        pn = torch.empty(2 * N, dtype=torch.float64, device=dev)
        C.sampled_norms(N, d, idx, refv, out, pn)
        pv = pn.cpu().numpy()
        parity = {"max_rel_l2": max(math.sqrt(pv[2 * i] / pv[2 * i + 1]) for i in range(N)),
                  "outputs": int(ok.sum()) * N, "kappa_M": info["kappa_M"],
                  "fp64_reliable": bool(info["fp64_reliable"]),
                  "note": "the GPU line's outputs against the fp64 oracle of cpu_baseline on the same plan and "
                          "inputs, at its kept positions; squared sums by K5 (cerar_sampled_norms)"}
        if not info["fp64_reliable"]:
            parity["note"] += ("; the plan is singular even in fp64 (fp64_reliable = 0), so the oracle's own "
                               "output is not meaningful and this figure is reported only")
        log(f"parity vs oracle: {parity['max_rel_l2']:.3g} over {parity['outputs']} outputs"
            + ("" if info["fp64_reliable"] else " (plan singular in fp64: reported only)"))

    step_bytes = N * C.algorithmic_bytes_per_worker(N, c, p)
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    result = {
        "metric": METRIC if args.workload == synth.HEADLINE else
                  f"encode+round+decode GB/s per worker (% HBM peak), N={N} c={c} d={d} fp32",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "workload_name": args.workload, "N": N, "c": c, "d": d, "p": p, "L": L,
                   "plan": plan_desc, "pct_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
                   "bytes_per_step": step_bytes, "encode": "out of place (grads kept for every step)"},
        "roofline": roofline,
        "kernels": kernels,
        "ms_per_step_with_events": round(ms_events, 4),
        "step_ms_events": step_spans,
        "bucketed": bucketed,
        "fused_variant": fused,
        "in_place_encode": in_place,
        "encode_spread": spread,
        "copy_gbps": round(copy_gbps, 1),
        "approx_rel_err_max": max(rel_err),
        "parity_vs_oracle": parity,
        "plan_info": {k: info[k] for k in ("kappa_M", "kappa_U", "kappa_R", "phi", "phi_closed_form",
                                            "comm_rate", "storage_rate", "r_star", "fp64_reliable")},
    }
    del grads, work, ws, out
    torch.cuda.empty_cache()
    if cpu is not None:
        result["cpu_baseline"] = cpu
    for k, v in list(result["plan_info"].items()):
        if isinstance(v, float) and not math.isfinite(v):
            result["plan_info"][k] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
