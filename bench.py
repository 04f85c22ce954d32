#!/usr/bin/env python3
"""Benchmark of the serving-simulation sweep on one MI355X.

One step = one whole sweep (every design point simulated to completion:
intake, block reservation / preemption, admission, roofline pricing and
state advance for every iteration, then the percentile statistics) with
traces and design points already resident in HBM.  Prints one JSON line.

The default workload is the largest sweep: 65536 design points x 10000
requests (7B GQA model, chunked prefill 256..2048, long-context prompt
mixture, bursty arrivals), generated from fixed seeds.

roofline: the simulation is bound by instruction issue (integer scheduling
and a short fp64 roofline per iteration; no dense contraction, negligible HBM
traffic).  ``achieved`` is the algorithmic VALU instruction count of the
dominant simulation launch divided by its HIP-event duration, with
  U = 6.5 wave64 VALU instructions per simulated iteration,
what one steady iteration costs in the kernels' cheapest path: iterations
priced up to 64 at a time, one per lane, in blocks (measured with the
SQ_INSTS_VALU counter on the u1 workload, 64 decodes with long outputs per
point, where almost every iteration is such a one: 6.7 per iteration,
rounded down).  Scheduling events (admissions, finishes, prefill
completions, preemptions) are not counted, so the fraction is the share of
the issue peak the sweep would use if every iteration cost as little as a
steady one.  Peak = 256 CUs x 4 SIMDs x 2.4 GHz / 4 cycles per wave64
instruction = 614.4 G instructions/s.  Every launch gets the same figure in
``roofline_launches`` (iterations it simulated to completion, from the
library's per-launch counters).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "simulated requests/sec across sweep on 1 MI355X; % VALU-issue peak"
VALU_ISSUE_PEAK = 256 * 4 * 2.4e9 / 4.0   # wave64 VALU instructions per second
U_ITER = 6.5
# simulation launches, 3 * stage + class (stages: one-worker points, prefill
# devices, decode devices of disaggregated points; register-chunk classes
# 1, 2, 4), named as rocprofv3 names the kernels
KERNEL_NAMES = tuple("sim_kernel<%d,%d>" % (c, st) for st in range(3) for c in (1, 2, 4))


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sim_kernel_traffic_c5.md")
# the sources whose change invalidates the recorded traffic counters
KERNEL_SOURCES = ("paper_2503_08415_amd/csrc/sim_kernel.hip",
                  "paper_2503_08415_amd/csrc/sweep_internal.h",
                  "paper_2503_08415_amd/csrc/host.hip",
                  "paper_2503_08415_amd/build.py")  # the compiler flags


def workloads_configs():
    from paper_2503_08415_amd import workloads
    return workloads.CONFIGS.keys()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(config, kernel):
    """HBM bytes per launch of ``kernel`` from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE summary, or None when it is missing or the kernel sources have
    changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            lines = f.read().splitlines()
    except OSError:
        return None
    sha, found = None, None
    for ln in lines:
        w = ln.strip().strip("`").split()
        if len(w) == 2 and w[0] == "sources-sha256:":
            sha = w[1]
        if len(w) == 4 and w[0] == "traffic-bytes:" and w[1] == config and w[2] == kernel:
            found = float(w[3])
    if sha is None or found is None or sha != kernel_sources_sha256():
        return None
    return found


def algorithmic_instructions(out):
    return U_ITER * out["n_iters"].astype(np.float64)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(model, traces, points, target_s, seed=0):
    """The oracle on a bounded, seeded sample of the same design points.

    Returns the baseline record and (sample indices, oracle point results),
    which the caller compares with the GPU's results for those points."""
    from oracle import tso
    from paper_2503_08415_amd import workloads
    n_points = len(points["peak_flops"])
    cores = tso.default_threads()
    rng = np.random.default_rng(seed)
    order = rng.permutation(n_points)
    # calibrate on a first slice, then size the sample to about target_s
    first = order[:max(cores, 8)]
    t0 = time.perf_counter()
    tso.run_points(model, traces, workloads.subset_points(points, first), n_threads=cores)
    dt = time.perf_counter() - t0
    per_point = dt / len(first)
    n_more = int(max(0, min(n_points - len(first), target_s / max(per_point, 1e-6))))
    sample = order[:len(first) + n_more]
    sub = workloads.subset_points(points, sample)
    t0 = time.perf_counter()
    out, _ = tso.run_points(model, traces, sub, n_threads=cores)
    dt = time.perf_counter() - t0
    n_req = int(sum(len(traces[int(t)]["arrival_ns"]) for t in sub["trace_id"]))
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = os.cpu_count() or 1
    rec = {"value": n_req / dt, "unit": "simulated requests/s", "cores": cores,
           "kind": "oracle",
           "sample": "%d of %d design points (seeded random), %d simulated requests, %.1f s wall"
                     % (len(sample), n_points, n_req, dt),
           "cpu_model": cpu_model(), "host_cores": os.cpu_count(), "affinity_cores": affinity,
           "threads_note": "one thread per design point at a time, on min(affinity cores, 16)"
                           " threads: one GPU's share of the host"}
    return rec, (sample, out)


def parity_of(gpu_out, sample, oracle_out):
    """Field-by-field comparison of the GPU's point results with the
    oracle's on the sampled points (used_block_ns within 1e-9 relative)."""
    g = gpu_out[sample]
    bad = np.zeros(len(sample), dtype=bool)
    fields = []
    for f in oracle_out.dtype.names:
        if f == "used_block_ns":
            ne = ~np.isclose(g[f], oracle_out[f], rtol=1e-9, atol=0.0)
        else:
            ne = g[f] != oracle_out[f]
        if ne.any():
            fields.append(f)
        bad |= ne
    return {"points": int(len(sample)), "mismatches": int(bad.sum()), "fields": fields,
            "run": "the last timed step's results"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="c5", choices=sorted(workloads_configs()))
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall time budget of the oracle baseline sample (0 = skip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run 8 plain device copies of BYTES bytes (reference for the "
                         "FETCH_SIZE / WRITE_SIZE traffic counters) and exit")
    args = ap.parse_args()
    if args.copy_calibration > 0:
        import torch
        src = torch.ones(args.copy_calibration, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(8):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": args.copy_calibration, "copies": 8}))
        return
    if args.gpus != 1:
        print("bench.py runs on one GPU: the sweep's design points are independent and the "
              "benchmark measures one GPU's share; --gpus %d is not supported" % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2503_08415_amd import sweep, workloads

    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    model, traces, points = workloads.make_config(args.config)
    n_points = len(points["peak_flops"])
    n_req = int(sum(len(traces[int(t)]["arrival_ns"]) for t in points["trace_id"]))
    digest = workloads.digests(model, traces, points)
    pinned = None
    try:
        with open(os.path.join(ROOT, "tests", "golden", "workload_sha256.json")) as f:
            pinned = json.load(f)["configs"].get(args.config) == digest
    except OSError:
        pass
    log("workload %s: %d points, %d simulated requests (generated in %.1fs)"
        % (args.config, n_points, n_req, time.perf_counter() - t0))
    sw = sweep.Sweep(model, traces, points)
    stream = torch.cuda.current_stream()

    for i in range(args.warmup):
        t0 = time.perf_counter()
        sw.run(stream)
        torch.cuda.synchronize()
        log("warmup %d: %.3fs" % (i, time.perf_counter() - t0))

    step_s, sim_ms, stats_ms, kms, kwork = [], [], [], [], []
    torch.cuda.synchronize()
    t_all = time.perf_counter()
    for i in range(args.steps):
        t0 = time.perf_counter()
        sw.run(stream)
        torch.cuda.synchronize()
        step_s.append(time.perf_counter() - t0)
        a, b = sw.timing()
        sim_ms.append(a)
        stats_ms.append(b)
        kms.append([k[0] for k in sw.kernel_timing()])
        kwork.append(sw.kernel_work())
        log("step %d: %.3fs (simulation %.1f ms, statistics %.1f ms, kernels %s)"
            % (i, step_s[-1], a, b, ["%.1f" % x for x in kms[-1]]))
    torch.cuda.synchronize()
    total_s = time.perf_counter() - t_all
    t0 = time.perf_counter()
    out, _ = sw.results()
    results_s = time.perf_counter() - t0
    sw.close()

    ms_per_step = 1e3 * total_s / args.steps
    value = n_req / (total_s / args.steps)
    status = np.bincount(out["status"], minlength=4).tolist()

    # roofline of every simulation launch from the iterations it simulated to
    # completion (a point handed from the 64-slot launch to a wider one counts
    # only where it completed; a disaggregated point's iterations are those of
    # its devices, each counted in its own stage's launch); the line's
    # roofline is the dominant launch's (longest mean duration)
    kmean = np.mean(np.array(kms), axis=0)
    w = algorithmic_instructions(out)
    work = np.array(kwork[-1], dtype=np.float64)
    launches = []
    for i in range(len(kmean)):
        if kmean[i] <= 0 and work[i] == 0:
            continue
        a_i = U_ITER * work[i] / (kmean[i] * 1e-3) if kmean[i] > 0 else 0.0
        launches.append({"kernel": KERNEL_NAMES[i], "iterations": int(work[i]),
                         "kernel_ms": float(kmean[i]), "achieved": a_i / 1e9,
                         "frac": a_i / VALU_ISSUE_PEAK})
    k = int(np.argmax(kmean))
    name, w_k, k_ms = KERNEL_NAMES[k], U_ITER * float(work[k]), float(kmean[k])
    traffic = recorded_traffic(args.config, name)
    achieved = w_k / (k_ms * 1e-3)
    roofline = {"bound": "alu", "achieved": achieved / 1e9, "peak": VALU_ISSUE_PEAK / 1e9,
                "unit": "G wave64 VALU instr/s", "frac": achieved / VALU_ISSUE_PEAK,
                "traffic": traffic, "kernel": name, "algorithmic_instr": w_k, "kernel_ms": k_ms}

    line = {
        "metric": METRIC, "value": value, "unit": "simulated requests/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int32/int64 + f64", "data": "synthetic",
        "config": {"workload": "%s: %s" % (args.config, workloads.CONFIGS[args.config][2]),
                   "design_points": n_points, "simulated_requests": n_req,
                   "model": "none (simulated transformer shape)",
                   "parallelism": "one wave64 workgroup per design point"},
        "workload_sha256": {"traces": digest["traces"], "points": digest["points"],
                            "matches_committed": pinned},
        "roofline": roofline,
        "roofline_launches": launches,
        "kernels_ms": {KERNEL_NAMES[i]: float(kmean[i]) for i in range(len(kmean))
                       if kmean[i] > 0},
        "simulation_phase_ms": float(np.mean(sim_ms)), "statistics_ms": float(np.mean(stats_ms)),
        "results_copy_ms": 1e3 * results_s,
        "frac_step": float(w.sum()) / (ms_per_step * 1e-3) / VALU_ISSUE_PEAK,
        "simulated_iterations": int(out["n_iters"].sum()),
        "simulated_iterations_by_kernel": {KERNEL_NAMES[i]: int(work[i])
                                           for i in range(len(work)) if work[i] > 0},
        "point_status_counts": status,
    }
    parity_ok = True
    if args.cpu_seconds > 0:
        log("cpu baseline: oracle on a sample (~%.0fs)..." % args.cpu_seconds)
        line["cpu_baseline"], (sample, o_out) = cpu_baseline(model, traces, points,
                                                             args.cpu_seconds)
        line["parity"] = parity_of(out, sample, o_out)
        parity_ok = line["parity"]["mismatches"] == 0
    print(json.dumps(line), flush=True)
    if not parity_ok:
        log("PARITY FAILURE: %d of %d sampled points differ from the oracle (%s)"
            % (line["parity"]["mismatches"], line["parity"]["points"],
               ", ".join(line["parity"]["fields"])))
        sys.exit(1)


if __name__ == "__main__":
    main()
