"""Seeded synthetic workloads for the serving-simulation sweep.

This module only *generates inputs*: request traces (arrival time, prompt
length, output length), transformer shapes and design-point grids.  It holds
none of the simulation's arithmetic (no block budgets, no cost model, no
scheduling), so both the HIP path and the CPU oracle can be fed the very same
bytes from it without sharing any of the method.

The paper drives its simulator with requests built from a dataset or from
parameters for distribution and rate (Sec. III, system overview) and measures
on ShareGPT (Sec. III-C, Sec. IV-A).  No dataset is used here: seeded
lognormal / uniform length laws with Poisson or bursty-Poisson arrivals stand
in for those workloads.

Generator rules (all configs):
  * ``numpy.random.Generator(PCG64(seed))`` with
    ``seed = 1_000_000 * config + 1_000 * replicate + rate_index``;
  * draw order: inter-arrival gaps, then prompt lengths, then output lengths;
  * arrivals are the cumulative fp64 sum of the gaps (first arrival = first
    gap), converted with ``floor(seconds * 1e9)`` to int64 nanoseconds;
  * lognormal lengths are rounded with ``rint`` and clipped; uniform integer
    ranges are inclusive;
  * bursty arrivals: the rate is ``lo`` on [0, P), ``hi`` on [P, 2P), ... ; a
    gap that would cross a phase boundary restarts at the boundary with the
    new rate (exact for a memoryless process);
  * mixture prompts: component uniforms first, then all lognormal draws, then
    all uniform-integer draws, then select;
  * one-trace-per-point sweeps seed point i's trace with
    ``1_000_000_000 + 1_000_000 * config + i`` (above every other seed).
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "MODELS", "CONFIGS", "make_trace", "make_config", "POINT_FIELDS",
    "FLOPS_GRID8", "BW_GRID8", "C4_CAPS", "digests",
]

# Transformer shapes (LLaMA-family layouts; the paper validates on
# LLaMA2-7B, Sec. III-C).  fp16 weights and KV (2 bytes per element).
MODELS = {
    # 32 layers, d=4096, 32 heads, MHA, gated FFN 11008, vocab 32000
    "llama2-7b": dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32,
                      ffn_dim=11008, ffn_gated=1, vocab=32000, w_bytes=2,
                      kv_bytes=2, weights_in_capacity=1),
    # 40 layers, d=5120, 40 heads, MHA, gated FFN 13824
    "llama2-13b": dict(n_layers=40, d_model=5120, n_heads=40, n_kv_heads=40,
                       ffn_dim=13824, ffn_gated=1, vocab=32000, w_bytes=2,
                       kv_bytes=2, weights_in_capacity=1),
    # 80 layers, d=8192, 64 query heads, 8 KV heads (GQA), gated FFN 28672.
    # Capacity is read as the per-GPU KV budget (weights not counted).
    "llama2-70b-kvonly": dict(n_layers=80, d_model=8192, n_heads=64,
                              n_kv_heads=8, ffn_dim=28672, ffn_gated=1,
                              vocab=32000, w_bytes=2, kv_bytes=2,
                              weights_in_capacity=0),
    # 32 layers, d=4096, 32 query heads, 8 KV heads (GQA), gated FFN 14336
    "gqa-7b": dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=8,
                   ffn_dim=14336, ffn_gated=1, vocab=32000, w_bytes=2,
                   kv_bytes=2, weights_in_capacity=1),
}

# 8-value hardware grids: FLOP/s = 100e12 * 25**(i/7), B/s = 1e12 * 10**(i/7).
# Written out as exact doubles so no libm difference can change a design point.
FLOPS_GRID8 = (100000000000000.0, 158381960876657.9, 250848455311351.97,
               397298702350926.1, 629249475320913.2, 996617657819344.2,
               1578462588897297.8, 2500000000000000.0)
BW_GRID8 = (1000000000000.0, 1389495494373.1377, 1930697728883.25,
            2682695795279.7256, 3727593720314.94, 5179474679231.212,
            7196856730011.52, 10000000000000.0)
# 32 capacities round(24e9 + i * 136e9 / 31), i < 32 (24 GB .. 160 GB)
C4_CAPS = tuple(int(round(24e9 + i * 136e9 / 31)) for i in range(32))

POINT_FIELDS = ("peak_flops", "mem_bw", "capacity_bytes", "mem_util_permille",
                "block_size", "max_batch", "chunk_size", "trace_id", "policy",
                "admit_mem_permille", "swap_overlap", "swap_bw", "n_prefill", "n_decode",
                "p_peak_flops", "p_mem_bw", "p_capacity_bytes", "kv_link_bw")

_NS = 1e9


def _seed(config: int, replicate: int, rate_index: int) -> int:
    return 1_000_000 * config + 1_000 * replicate + rate_index


def _poisson_arrivals(rng, n, rate):
    gaps = rng.exponential(1.0 / rate, size=n)
    return np.cumsum(gaps)


def _bursty_arrivals(rng, n, lo, hi, period):
    out = np.empty(n, dtype=np.float64)
    t = 0.0
    for i in range(n):
        while True:
            phase = int(t // period)
            rate = lo if phase % 2 == 0 else hi
            end = (phase + 1) * period
            g = rng.standard_exponential() / rate
            if t + g < end:
                t = t + g
                break
            t = float(end)
        out[i] = t
    return out


def _lognormal_int(rng, n, mu, sigma, lo, hi):
    x = np.rint(rng.lognormal(mu, sigma, size=n))
    return np.clip(x, lo, hi).astype(np.int32)


def _uniform_int(rng, n, lo, hi):
    return rng.integers(lo, hi, size=n, endpoint=True).astype(np.int32)


def make_trace(spec: dict, n: int, seed: int) -> dict:
    """Build one request trace.

    ``spec`` keys: ``arrival`` = ("poisson", rate) | ("bursty", lo, hi, period_s);
    ``prompt`` / ``output`` = ("uniform", lo, hi) | ("lognormal", mu, sigma,
    lo, hi) | ("mixture", w, ("lognormal", ...), ("uniform", ...)).
    Returns int64 ``arrival_ns`` (non-decreasing), int32 ``prompt_len`` and
    int32 ``output_len``, each of length ``n``.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    arr = spec["arrival"]
    if arr[0] == "poisson":
        secs = _poisson_arrivals(rng, n, float(arr[1]))
    elif arr[0] == "bursty":
        secs = _bursty_arrivals(rng, n, float(arr[1]), float(arr[2]), float(arr[3]))
    else:
        raise ValueError(arr)
    arrival_ns = np.floor(secs * _NS).astype(np.int64)

    def lengths(law):
        if law[0] == "uniform":
            return _uniform_int(rng, n, law[1], law[2])
        if law[0] == "lognormal":
            return _lognormal_int(rng, n, *law[1:])
        if law[0] == "mixture":
            w, first, second = law[1], law[2], law[3]
            pick_first = rng.random(n) < w
            assert first[0] == "lognormal" and second[0] == "uniform"
            a = _lognormal_int(rng, n, *first[1:])
            b = _uniform_int(rng, n, second[1], second[2])
            return np.where(pick_first, a, b).astype(np.int32)
        raise ValueError(law)

    prompt = lengths(spec["prompt"])
    output = lengths(spec["output"])
    return {"arrival_ns": arrival_ns, "prompt_len": prompt, "output_len": output}


_LN_P_C2 = ("lognormal", 5.5, 1.0, 4, 4096)
_LN_O_C2 = ("lognormal", 5.0, 0.9, 1, 2048)


def _points(rows):
    pts = {k: [] for k in POINT_FIELDS}
    for r in rows:
        for k in POINT_FIELDS:
            pts[k].append(r.get(k, 0))
    return {
        "peak_flops": np.asarray(pts["peak_flops"], dtype=np.float64),
        "mem_bw": np.asarray(pts["mem_bw"], dtype=np.float64),
        "capacity_bytes": np.asarray(pts["capacity_bytes"], dtype=np.int64),
        "mem_util_permille": np.asarray(pts["mem_util_permille"], dtype=np.int32),
        "block_size": np.asarray(pts["block_size"], dtype=np.int32),
        "max_batch": np.asarray(pts["max_batch"], dtype=np.int32),
        "chunk_size": np.asarray(pts["chunk_size"], dtype=np.int32),
        "trace_id": np.asarray(pts["trace_id"], dtype=np.int32),
        "policy": np.asarray(pts["policy"], dtype=np.int32),
        "admit_mem_permille": np.asarray(pts["admit_mem_permille"], dtype=np.int32),
        "swap_overlap": np.asarray(pts["swap_overlap"], dtype=np.int32),
        "swap_bw": np.asarray(pts["swap_bw"], dtype=np.float64),
        "n_prefill": np.asarray(pts["n_prefill"], dtype=np.int32),
        "n_decode": np.asarray(pts["n_decode"], dtype=np.int32),
        "p_peak_flops": np.asarray(pts["p_peak_flops"], dtype=np.float64),
        "p_mem_bw": np.asarray(pts["p_mem_bw"], dtype=np.float64),
        "p_capacity_bytes": np.asarray(pts["p_capacity_bytes"], dtype=np.int64),
        "kv_link_bw": np.asarray(pts["kv_link_bw"], dtype=np.float64),
    }


def _c1(n_req):
    spec = {"arrival": ("poisson", 2.0), "prompt": ("uniform", 16, 256),
            "output": ("uniform", 8, 128)}
    traces = [make_trace(spec, n_req, _seed(1, 0, 0))]
    rows = [dict(peak_flops=312e12, mem_bw=2.0e12, capacity_bytes=80_000_000_000,
                 mem_util_permille=900, block_size=16, max_batch=32,
                 chunk_size=0, trace_id=0)]
    return "llama2-7b", traces, rows


def _c2(n_req):
    traces = []
    for r in range(16):
        spec = {"arrival": ("poisson", float(r + 1)), "prompt": _LN_P_C2,
                "output": _LN_O_C2}
        traces.append(make_trace(spec, n_req, _seed(2, 0, r)))
    rows = []
    for r in range(16):
        for f in (200e12, 400e12, 800e12, 1600e12):
            for bw in (1e12, 2e12, 4e12, 8e12):
                rows.append(dict(peak_flops=f, mem_bw=bw,
                                 capacity_bytes=80_000_000_000,
                                 mem_util_permille=900, block_size=16,
                                 max_batch=64, chunk_size=0, trace_id=r))
    return "llama2-7b", traces, rows


_CAPS4 = (40_000_000_000, 80_000_000_000, 192_000_000_000, 288_000_000_000)


def _c3(n_req):
    traces = []
    for k in range(4):
        spec = {"arrival": ("poisson", 8.0), "prompt": _LN_P_C2, "output": _LN_O_C2}
        traces.append(make_trace(spec, n_req, _seed(3, k, 0)))
    rows = []
    for k in range(4):
        for f in FLOPS_GRID8:
            for bw in BW_GRID8:
                for cap in _CAPS4:
                    for b in (8, 16):
                        for m in (64, 256):
                            rows.append(dict(peak_flops=f, mem_bw=bw,
                                             capacity_bytes=cap,
                                             mem_util_permille=900,
                                             block_size=b, max_batch=m,
                                             chunk_size=0, trace_id=k))
    return "llama2-13b", traces, rows


def _c4(n_req):
    traces = []
    for r in range(8):
        spec = {"arrival": ("poisson", 4.0 * (r + 1)),
                "prompt": ("lognormal", 6.0, 1.1, 4, 8192),
                "output": ("lognormal", 5.3, 1.0, 1, 4096)}
        traces.append(make_trace(spec, n_req, _seed(4, 0, r)))
    rows = []
    for r in range(8):
        for cap in C4_CAPS:
            for f in FLOPS_GRID8:
                for bw in BW_GRID8:
                    rows.append(dict(peak_flops=f, mem_bw=bw, capacity_bytes=cap,
                                     mem_util_permille=1000, block_size=16,
                                     max_batch=256, chunk_size=0, trace_id=r))
    return "llama2-70b-kvonly", traces, rows


def _c5(n_req):
    traces = []
    for k in range(16):
        spec = {"arrival": ("bursty", 2.0, 20.0, 60.0),
                "prompt": ("mixture", 0.7, ("lognormal", 6.0, 1.0, 4, 8192),
                           ("uniform", 8192, 32768)),
                "output": _LN_O_C2}
        traces.append(make_trace(spec, n_req, _seed(5, k, 0)))
    rows = []
    for k in range(16):
        for chunk in (256, 512, 1024, 2048):
            for f in FLOPS_GRID8:
                for bw in BW_GRID8:
                    for cap in _CAPS4:
                        for b in (8, 16):
                            for m in (64, 256):
                                rows.append(dict(peak_flops=f, mem_bw=bw,
                                                 capacity_bytes=cap,
                                                 mem_util_permille=900,
                                                 block_size=b, max_batch=m,
                                                 chunk_size=chunk, trace_id=k))
    return "gqa-7b", traces, rows


def _c6(n_req, reps=1):
    """Scheduling policies and the admission memory ratio under memory
    pressure (the studies of Sec. IV-A and Sec. IV-B): 16 arrival rates x
    3 policies x 4 ratios x 2 small capacities, 7B model, unchunked; reps
    replicates with their own traces (replicate 0 is the base sweep)."""
    traces, rows = [], []
    for rep in range(reps):
        base = len(traces)
        for r in range(16):
            spec = {"arrival": ("poisson", float(r + 1)), "prompt": _LN_P_C2,
                    "output": _LN_O_C2}
            traces.append(make_trace(spec, n_req, _seed(6, rep, r)))
        for r in range(16):
            for policy in (0, 1, 2):
                for ratio in (0, 600, 800, 950):
                    for cap in (24_000_000_000, 40_000_000_000):
                        rows.append(dict(peak_flops=312e12, mem_bw=2e12, capacity_bytes=cap,
                                         mem_util_permille=900, block_size=16, max_batch=64,
                                         chunk_size=0, trace_id=base + r, policy=policy,
                                         admit_mem_permille=ratio))
    return "llama2-7b", traces, rows


def _c7(n_req, reps=1):
    """Preemption by recompute against preemption by swap (Sec. IV-B; the
    transfer priced by the communication model of Sec. III-B) under memory
    pressure: 16 arrival rates x {recompute, swap over 16 / 32 / 64 GB/s
    after the compute, swap over 64 GB/s overlapping it} x {20, 24} GB x
    {unchunked, chunk 512}, 7B model; reps replicates with their own traces."""
    traces, rows = [], []
    for rep in range(reps):
        base = len(traces)
        for r in range(16):
            spec = {"arrival": ("poisson", float(r + 1)), "prompt": _LN_P_C2,
                    "output": _LN_O_C2}
            traces.append(make_trace(spec, n_req, _seed(7, rep, r)))
        for r in range(16):
            for bw, overlap in ((0.0, 0), (16e9, 0), (32e9, 0), (64e9, 0), (64e9, 1)):
                for cap in (20_000_000_000, 24_000_000_000):
                    for chunk in (0, 512):
                        rows.append(dict(peak_flops=312e12, mem_bw=2e12, capacity_bytes=cap,
                                         mem_util_permille=900, block_size=16, max_batch=64,
                                         chunk_size=chunk, trace_id=base + r, swap_bw=bw,
                                         swap_overlap=overlap))
    return "llama2-7b", traces, rows


def _c8(n_req, reps=1):
    """Disaggregated prefill and decode on an 8-device node (Sec. V: the best
    prefill-to-decode device ratio over input and output lengths, and the
    prefill device's compute, capacity and bandwidth): 4 length mixes
    (lognormal prompts around 128 or 1024 tokens x outputs around 128 or
    512) x 4 arrival rates x P/D splits {1/7, 2/6, 3/5, 4/4} x prefill
    hardware {A100-like, 2x FLOP/s, 1/4 capacity, 1/4 bandwidth}, 7B model,
    decode devices A100-like, KV links of 25 GB/s; reps replicates with
    their own traces (replicate slot of the seed: 4 * rep + mix)."""
    mixes = [(4.85, 4.85), (4.85, 6.2), (6.9, 4.85), (6.9, 6.2)]  # log-means: ~128, ~512, ~1024
    rates = (5.0, 10.0, 20.0, 40.0)
    prefill_hw = [(312e12, 2e12, 80_000_000_000), (624e12, 2e12, 80_000_000_000),
                  (312e12, 2e12, 20_000_000_000), (312e12, 0.5e12, 80_000_000_000)]
    traces, rows = [], []
    for rep in range(reps):
        base = len(traces)
        for m, (lp, lo) in enumerate(mixes):
            for r, rate in enumerate(rates):
                spec = {"arrival": ("poisson", rate),
                        "prompt": ("lognormal", lp, 0.6, 4, 8192),
                        "output": ("lognormal", lo, 0.6, 1, 4096)}
                traces.append(make_trace(spec, n_req, _seed(8, 4 * rep + m, r)))
        for k in range(len(mixes) * len(rates)):
            for n_p in (1, 2, 3, 4):
                for pf, pb, pc in prefill_hw:
                    rows.append(dict(peak_flops=312e12, mem_bw=2e12,
                                     capacity_bytes=80_000_000_000, mem_util_permille=900,
                                     block_size=16, max_batch=64, chunk_size=0,
                                     trace_id=base + k, n_prefill=n_p, n_decode=8 - n_p,
                                     p_peak_flops=pf, p_mem_bw=pb, p_capacity_bytes=pc,
                                     kv_link_bw=25e9))
    return "llama2-7b", traces, rows


def _c4u(n_req):
    """c4's grid with one trace per design point (trace_id = point): every
    point reads its own 4000 records, so the sweep streams 1.05 GB of distinct
    trace bytes from HBM.  Point i draws its trace at its row's rate with
    seed 1_000_000_000 + 1_000_000 * 4 + i."""
    _, _, rows = _c4(0)
    traces = []
    for i, row in enumerate(rows):
        rate = 4.0 * (row["trace_id"] + 1)
        spec = {"arrival": ("poisson", rate),
                "prompt": ("lognormal", 6.0, 1.1, 4, 8192),
                "output": ("lognormal", 5.3, 1.0, 1, 4096)}
        traces.append(make_trace(spec, n_req, 1_000_000_000 + 1_000_000 * 4 + i))
        row["trace_id"] = i
    return "llama2-70b-kvonly", traces, rows


def _u1(n_req):
    """Calibration of the steady path: 8192 identical points, each 64
    requests arriving together (prompt 16, output 4000) that decode side by
    side, so almost every iteration is a steady one in a long block.  Their
    KV does not all fit (6976 blocks of 16 tokens), so block shortages
    preempt some of them: about 6300 iterations per point."""
    n = 64
    traces = [{"arrival_ns": np.zeros(n, np.int64), "prompt_len": np.full(n, 16, np.int32),
               "output_len": np.full(n, 4000, np.int32)}]
    rows = [dict(peak_flops=312e12, mem_bw=2e12, capacity_bytes=80_000_000_000,
                 mem_util_permille=900, block_size=16, max_batch=64, chunk_size=0,
                 trace_id=0) for _ in range(8192)]
    return "llama2-7b", traces, rows


# name -> (builder, default requests per trace, description)
CONFIGS = {
    "c1": (_c1, 64, "1 point x 64 requests, 7B MHA, 312 TF / 2 TB/s / 80 GB, "
                    "block 16, max batch 32"),
    "c2": (_c2, 1000, "256 points x 1000 requests, 7B MHA, 16 rates x 4 FLOP/s x 4 BW, "
                      "80 GB, block 16, max batch 64"),
    "c3": (_c3, 2000, "4096 points x 2000 requests, 13B MHA, 8 FLOP/s x 8 BW x 4 cap "
                      "x 2 block x 2 max batch x 4 seeds"),
    "c4": (_c4, 4000, "16384 points x 4000 requests, 80-layer GQA, KV-only capacity "
                      "24-160 GB, 8 rates x 32 caps x 8 FLOP/s x 8 BW, max batch 256"),
    "c5": (_c5, 10000, "65536 points x 10000 requests, 7B GQA, chunked prefill "
                       "{256..2048}, long-context mixture, bursty arrivals"),
    "c6": (_c6, 2000, "384 points x 2000 requests, 7B MHA, 16 rates x {mixed, prefill-first, "
                      "static} x admission ratio {off, 60%, 80%, 95%} x {24, 40} GB"),
    "c7": (_c7, 2000, "320 points x 2000 requests, 7B MHA, 16 rates x {recompute, swap "
                      "16/32/64 GB/s, swap 64 GB/s overlapped} x {20, 24} GB x {no chunk, 512}"),
    "u1": (_u1, 64, "8192 points x 64 requests decoding together, output 4000 "
                    "(calibration of the steady path)"),
    "c8": (_c8, 2000, "256 disaggregated points x 2000 requests, 7B MHA, 4 length mixes x "
                      "4 rates x P/D {1/7, 2/6, 3/5, 4/4} x 4 prefill devices, 25 GB/s KV links"),
    # the same studies at a size that fills the GPU (at least 8192 simulation
    # units: one per one-worker point, one per device of a disaggregated one)
    "c6x": (lambda n: _c6(n, 24), 2000, "9216 points x 2000 requests: c6 with 24 replicates "
                                        "(own traces each)"),
    "c7x": (lambda n: _c7(n, 26), 2000, "8320 points x 2000 requests: c7 with 26 replicates "
                                        "(own traces each)"),
    "c8x": (lambda n: _c8(n, 4), 2000, "1024 disaggregated points (8192 devices) x 2000 "
                                       "requests: c8 with 4 replicates (own traces each)"),
    "c4u": (_c4u, 4000, "16384 points x 4000 requests: c4 with one trace per point "
                        "(1.05 GB of distinct trace records)"),
}


def make_config(name: str, n_requests: int | None = None):
    """Return ``(model_dict, traces, points)`` for a named sweep.

    ``traces`` is a list of dicts of arrays (see :func:`make_trace`);
    ``points`` is a dict of per-point arrays keyed by ``POINT_FIELDS``.
    ``n_requests`` overrides the per-trace request count (smaller parity
    cases use the same laws and seeds, truncated draws included).
    """
    builder, n_default, _ = CONFIGS[name]
    n = n_default if n_requests is None else int(n_requests)
    model_name, traces, rows = builder(n)
    return dict(MODELS[model_name]), traces, _points(rows)


def subset_points(points: dict, idx) -> dict:
    """Select design points by index (same field layout)."""
    idx = np.asarray(idx, dtype=np.int64)
    return {k: np.ascontiguousarray(v[idx]) for k, v in points.items()}


def digests(model: dict, traces, points: dict) -> dict:
    """SHA-256 of a workload's bytes: traces (arrival int64, prompt int32,
    output int32 per trace, little-endian, in trace order), the point grid
    (fields in sorted order) and the model shape (sorted JSON)."""
    import hashlib
    import json
    ht = hashlib.sha256()
    for tr in traces:
        ht.update(np.ascontiguousarray(tr["arrival_ns"], dtype="<i8").tobytes())
        ht.update(np.ascontiguousarray(tr["prompt_len"], dtype="<i4").tobytes())
        ht.update(np.ascontiguousarray(tr["output_len"], dtype="<i4").tobytes())
    hp = hashlib.sha256()
    for f in sorted(points):
        hp.update(f.encode())
        hp.update(np.ascontiguousarray(points[f]).tobytes())
    hm = hashlib.sha256(json.dumps(model, sort_keys=True).encode())
    return {"traces": ht.hexdigest(), "points": hp.hexdigest(), "model": hm.hexdigest(),
            "n_traces": len(traces), "n_points": int(len(points["peak_flops"]))}
