"""Parity of the HIP sweep with the CPU oracle, through the C ABI.

Scheduling decisions, timestamps and every integer aggregate must match
bit for bit; the fp64 time integral of used blocks within 1e-9 relative.
The per-point digest hashes every finished / rejected request's record, so
matching digests cover per-request parity for points whose records are not
copied back.  Every GPU run carries an iteration cap derived from the
oracle so a scheduling bug ends as a mismatch, never as a hang.
"""
import json
import os
import sys
import time

import numpy as np
import pytest

from paper_2503_08415_amd import workloads as W

pytestmark = pytest.mark.gpu

GOLD = os.path.join(os.path.dirname(__file__), "golden")
REL_TOL = 1e-9


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2503_08415_amd import sweep
    sweep.lib()
    return sweep


def gpu_run(S, model, traces, points, per_request=False, **kw):
    # No wall-clock watchdog by default: the same code path as the benchmark,
    # whose steady stretches run to their first event.  Every call passes an
    # iteration cap (from the oracle where it has run), so a scheduling bug
    # ends as a mismatch, never as a hang.
    assert kw.get("iter_cap", 0) > 0, "every GPU run carries an iteration cap"
    kw.setdefault("point_time_limit_ms", 0)
    sw = S.Sweep(model, traces, points, per_request=per_request, **kw)
    try:
        sw.run()
        out, req = sw.results()
    finally:
        sw.close()
    return out, req


def compare_points(g, o, label=""):
    assert len(g) == len(o)
    bad = []
    for f in o.dtype.names:
        if f == "used_block_ns":
            ok = np.isclose(g[f], o[f], rtol=REL_TOL, atol=0.0)
        else:
            ok = g[f] == o[f]
        if not ok.all():
            idx = np.nonzero(~ok)[0]
            bad.append((f, int(idx.size), int(idx[0]), g[f][idx[0]], o[f][idx[0]]))
    assert not bad, "%s point mismatches (field, count, first, gpu, oracle): %s" % (label, bad[:8])


def compare_requests(g, o, label=""):
    assert g.shape == o.shape
    for f in o.dtype.names:
        ne = g[f] != o[f]
        if ne.any():
            p, r = [int(x[0]) for x in np.nonzero(ne)]
            raise AssertionError("%s request mismatch in %s at point %d request %d: gpu %s oracle %s"
                                 % (label, f, p, r, g[p, r], o[p, r]))


def cap_from(oracle_out):
    return int(oracle_out["n_iters"].max()) * 2 + 1000


FLOAT_FIELDS = ("peak_flops", "mem_bw", "swap_bw", "p_peak_flops", "p_mem_bw", "kv_link_bw")


def hand_sweep():
    with open(os.path.join(GOLD, "hand_traces.json")) as f:
        g = json.load(f)
    traces, rows = [], []
    for k, c in enumerate(g["cases"]):
        r = c["requests"]
        traces.append({"arrival_ns": np.array([x[0] for x in r], np.int64),
                       "prompt_len": np.array([x[1] for x in r], np.int32),
                       "output_len": np.array([x[2] for x in r], np.int32)})
        nb, b = c["num_blocks"], c["block_size"]
        rows.append(dict(peak_flops=1e300, mem_bw=1e300,
                         capacity_bytes=nb * b * 16 if nb > 0 else 1, mem_util_permille=1000,
                         block_size=b, max_batch=c["max_batch"], chunk_size=c["chunk_size"],
                         trace_id=k, policy=c.get("policy", 0),
                         admit_mem_permille=c.get("admit_mem_permille", 0),
                         swap_bw=c.get("swap_bw", 0.0), swap_overlap=c.get("swap_overlap", 0),
                         n_prefill=c.get("n_prefill", 0), n_decode=c.get("n_decode", 0),
                         p_peak_flops=1e300, p_mem_bw=1e300,
                         p_capacity_bytes=max(1, c.get("prefill_blocks", 0) * b * 16),
                         kv_link_bw=c.get("kv_link_bw", 0.0)))
    pts = {k: np.array([r[k] for r in rows]) for k in rows[0]}
    pts = {k: (v.astype(np.float64) if k in FLOAT_FIELDS else
               v.astype(np.int64) if k in ("capacity_bytes", "p_capacity_bytes") else
               v.astype(np.int32))
           for k, v in pts.items()}
    return g["model"], traces, pts, g["cases"]


def test_hand_traced_schedules_gpu(S, oracle):
    model, traces, pts, cases = hand_sweep()
    say("hand traces: %d cases" % len(cases))
    out, req = gpu_run(S, model, traces, pts, per_request=True, iter_cap=10_000)
    for k, c in enumerate(cases):
        n = len(c["requests"])
        got = [[int(x) for x in r] for r in req[k, :n].tolist()]
        assert got == c["expect_req"], c["name"]
        for f, v in c["expect_point"].items():
            assert out[k][f] == v, (c["name"], f)
    o_out, o_req = oracle.run_points(model, traces, pts, per_request=True)
    compare_points(out, o_out, "hand")
    compare_requests(req, o_req, "hand")


@pytest.mark.parametrize("name", ["c1", "c2"])
def test_full_config_per_request(S, oracle, name):
    m, traces, pts = W.make_config(name)
    say("%s: %d points, oracle..." % (name, len(pts["peak_flops"])))
    t0 = time.time()
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    say("%s: oracle %.1fs, gpu..." % (name, time.time() - t0))
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, name)
    compare_requests(req, o_req, name)
    assert (out["status"] == 0).all()


def _fuzz_case(rng, n_pts):
    traces, rows = [], []
    for k in range(n_pts):
        n = int(rng.integers(0, 41))
        gaps = rng.choice([0, 0, 1, 3, 50, 10_000], size=n)
        a = np.cumsum(gaps).astype(np.int64)
        p = rng.integers(1, 30, size=n).astype(np.int32)
        o = rng.integers(1, 12, size=n).astype(np.int32)
        traces.append({"arrival_ns": a, "prompt_len": p, "output_len": o})
        M = int(rng.choice([1, 2, 3, 5, 64, 65, 100, 130, 256]))
        b = int(rng.choice([1, 2, 3, 16]))
        K = int(rng.choice([0, 0, M, M + int(rng.integers(0, 9))]))
        nb = int(rng.integers(0, 21)) if M < 64 else int(rng.integers(0, 400))
        fast = rng.random() < 0.5
        policy = int(rng.choice([0, 0, 0, 1, 2]))  # mixed, prefill-first, static
        if policy == 1:
            K = 0
        permille = int(rng.choice([0, 0, 0, 250, 500, 1000]))
        # swap preemption over a link moving a 16-byte token in 16, 0.5 or 0.016 ns
        swap_bw = float(rng.choice([0.0, 0.0, 0.0, 1e9, 3.2e10, 1e12]))
        # a quarter of the points disaggregated: 1-3 prefill and 1-3 decode
        # devices, KV links moving a token in 0, 1 or 10 ns
        pd = dict(n_prefill=0, n_decode=0, p_peak_flops=0.0, p_mem_bw=0.0, p_capacity_bytes=0,
                  kv_link_bw=0.0)
        if rng.random() < 0.25:
            policy = 0
            nbp = int(rng.integers(0, 21)) if M < 64 else int(rng.integers(0, 400))
            pfast = rng.random() < 0.5
            pd = dict(n_prefill=int(rng.integers(1, 4)), n_decode=int(rng.integers(1, 4)),
                      p_peak_flops=1e300 if pfast else float(rng.choice([2e9, 5e9])),
                      p_mem_bw=1e300 if pfast else float(rng.choice([2e8, 1e9])),
                      p_capacity_bytes=max(1, nbp * b * 16),
                      kv_link_bw=float(rng.choice([0.0, 16e9, 1.6e9])))
        rows.append(dict(peak_flops=1e300 if fast else float(rng.choice([1e9, 3e9])),
                         mem_bw=1e300 if fast else float(rng.choice([1e8, 7e8])),
                         capacity_bytes=max(1, nb * b * 16), mem_util_permille=1000,
                         block_size=b, max_batch=M, chunk_size=K, trace_id=k,
                         policy=policy, admit_mem_permille=permille, swap_bw=swap_bw,
                         swap_overlap=int(rng.integers(0, 2)), **pd))
    pts = {
        "peak_flops": np.array([r["peak_flops"] for r in rows], np.float64),
        "mem_bw": np.array([r["mem_bw"] for r in rows], np.float64),
        "capacity_bytes": np.array([r["capacity_bytes"] for r in rows], np.int64),
        "p_capacity_bytes": np.array([r["p_capacity_bytes"] for r in rows], np.int64),
        **{f: np.array([r[f] for r in rows], np.float64)
           for f in ("swap_bw", "p_peak_flops", "p_mem_bw", "kv_link_bw")},
        **{f: np.array([r[f] for r in rows], np.int32)
           for f in ("mem_util_permille", "block_size", "max_batch", "chunk_size", "trace_id",
                     "policy", "admit_mem_permille", "swap_overlap", "n_prefill", "n_decode")}}
    return traces, pts


def test_fuzz_tiny_points(S, oracle):
    """Thousands of tiny random points: sequential oracle vs the kernel's
    prefix-scan formulation of reservation, preemption and admission."""
    model = {"n_layers": 1, "d_model": 8, "n_heads": 2, "n_kv_heads": 1, "ffn_dim": 16,
             "ffn_gated": 1, "vocab": 10, "w_bytes": 2, "kv_bytes": 2,
             "weights_in_capacity": 0}
    rng = np.random.default_rng(2024)
    total_pre = 0
    for rnd in range(12):
        traces, pts = _fuzz_case(rng, 1500)
        o_out, o_req = oracle.run_points(model, traces, pts, per_request=True)
        say("fuzz round %d: oracle preemptions %d" % (rnd, int(o_out["n_preempt"].sum())))
        out, req = gpu_run(S, model, traces, pts, per_request=True, iter_cap=cap_from(o_out))
        compare_points(out, o_out, "fuzz%d" % rnd)
        compare_requests(req, o_req, "fuzz%d" % rnd)
        total_pre += int(o_out["n_preempt"].sum())
    assert total_pre > 100


def test_full_c6_policies(S, oracle):
    """Static batching, prefill-first iterations and the admission memory
    ratio under memory pressure: every point, per request on a subset."""
    m, traces, pts = W.make_config("c6")
    t0 = time.time()
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    say("c6: oracle %.1fs, preemptions %d" % (time.time() - t0, int(o_out["n_preempt"].sum())))
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "c6")
    compare_requests(req, o_req, "c6")
    assert (out["status"] == 0).all()
    # the ratio keeps memory for running requests: fewer preemptions
    ratio = pts["admit_mem_permille"]
    assert out["n_preempt"][ratio == 600].sum() < out["n_preempt"][ratio == 0].sum()


def test_full_c7_swap(S, oracle):
    """Preemption by swap (transfers after the compute or overlapping it)
    against preemption by recompute under memory pressure: every point and
    every request."""
    m, traces, pts = W.make_config("c7")
    t0 = time.time()
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    say("c7: oracle %.1fs, preemptions %d" % (time.time() - t0, int(o_out["n_preempt"].sum())))
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "c7")
    compare_requests(req, o_req, "c7")
    assert (out["status"] == 0).all()
    swap = pts["swap_bw"] > 0
    assert out["n_preempt"][swap].sum() > 1000 and out["n_preempt"][~swap].sum() > 1000
    # transfers that overlap the compute never lengthen an iteration beyond
    # the sequential ones at the same bandwidth: lower mean latency overall
    fast = pts["swap_bw"] == 64e9
    ov, sq = fast & (pts["swap_overlap"] == 1), fast & (pts["swap_overlap"] == 0)
    assert out["sum_e2e_ns"][ov].sum() < out["sum_e2e_ns"][sq].sum()


def test_full_c8_disaggregated(S, oracle):
    """Disaggregated prefill and decode devices (P/D splits of an 8-device
    node, four prefill-device variants): every point and every request."""
    m, traces, pts = W.make_config("c8")
    t0 = time.time()
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    say("c8: oracle %.1fs, iterations %d" % (time.time() - t0, int(o_out["n_iters"].sum())))
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "c8")
    compare_requests(req, o_req, "c8")
    assert (out["status"] == 0).all()
    # first tokens come from the prefill side only: twice the prefill FLOP/s
    # never raises the TTFT sum
    hw = np.arange(len(pts["peak_flops"])) % 4
    assert (out["sum_ttft_ns"][hw == 1] <= out["sum_ttft_ns"][hw == 0]).all()


def _pd_rows(base, **kw):
    r = dict(base)
    r.update(kw)
    return r


def test_disaggregated_edges(S, oracle):
    """Disaggregated points at the edges: empty trace, no KV block on either
    side, the most devices, max batch 256 on both sides, chunked prefill,
    swap on the decode side, a sub-range of points and the iteration cap."""
    m = W.MODELS["llama2-7b"]
    rng = np.random.default_rng(7)
    n = 300
    tr = {"arrival_ns": np.sort(rng.integers(0, 5_000_000_000, n)).astype(np.int64),
          "prompt_len": rng.integers(1, 3000, n).astype(np.int32),
          "output_len": rng.integers(1, 400, n).astype(np.int32)}
    empty = {"arrival_ns": np.zeros(0, np.int64), "prompt_len": np.zeros(0, np.int32),
             "output_len": np.zeros(0, np.int32)}
    traces = [tr, empty]
    base = dict(peak_flops=312e12, mem_bw=2e12, capacity_bytes=80_000_000_000,
                mem_util_permille=900, block_size=16, max_batch=64, chunk_size=0, trace_id=0,
                policy=0, admit_mem_permille=0, swap_overlap=0, swap_bw=0.0, n_prefill=2,
                n_decode=3, p_peak_flops=500e12, p_mem_bw=1e12,
                p_capacity_bytes=40_000_000_000, kv_link_bw=20e9)
    rows = [
        _pd_rows(base, trace_id=1),                                    # empty trace
        _pd_rows(base, p_capacity_bytes=10_000_000_000),               # prefill side: no KV
        _pd_rows(base, capacity_bytes=10_000_000_000),                 # decode side: no KV
        _pd_rows(base, n_prefill=16, n_decode=16),                     # the most devices
        _pd_rows(base, max_batch=256, n_prefill=1, n_decode=1),        # class 2 on both sides
        _pd_rows(base, max_batch=100, chunk_size=512),                 # class 1, chunked
        _pd_rows(base, capacity_bytes=18_000_000_000, swap_bw=32e9,    # decode-side pressure,
                 admit_mem_permille=900, n_decode=1),                  # swap and the ratio
        _pd_rows(base, capacity_bytes=18_000_000_000, n_decode=1),     # ... with recompute
        _pd_rows(base, kv_link_bw=0.0, n_prefill=1),                   # instant link
        _pd_rows(base, n_prefill=0, n_decode=0),                       # one worker, same sweep
    ]
    pts = {k: np.array([r[k] for r in rows]) for k in rows[0]}
    pts = {k: (v.astype(np.float64) if k in FLOAT_FIELDS else
               v.astype(np.int64) if k in ("capacity_bytes", "p_capacity_bytes") else
               v.astype(np.int32)) for k, v in pts.items()}
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    assert (o_out["status"][[1, 2]] == 1).all() and o_out["n_preempt"][[6, 7]].min() > 0
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "pd edge")
    compare_requests(req, o_req, "pd edge")
    # a sub-range of the points
    sub = dict(first_point=3, n_points=4)
    out2, req2 = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out), **sub)
    compare_points(out2, o_out[3:7], "pd sub-range")
    compare_requests(req2, o_req[3:7], "pd sub-range")
    # the iteration cap stops each device alike
    o_cap, o_rq = oracle.run_points(m, traces, pts, per_request=True, iter_cap=50)
    g_cap, g_rq = gpu_run(S, m, traces, pts, per_request=True, iter_cap=50)
    compare_points(g_cap, o_cap, "pd iter cap")
    compare_requests(g_rq, o_rq, "pd iter cap")
    assert (g_cap["status"] == 2).sum() >= 5


def test_full_c3_points(S, oracle):
    m, traces, pts = W.make_config("c3")
    t0 = time.time()
    o_out, _ = oracle.run_points(m, traces, pts)
    say("c3: oracle %.1fs" % (time.time() - t0))
    out, _ = gpu_run(S, m, traces, pts, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "c3")
    # per-request records on a sub-range of points
    sub = dict(first_point=1000, n_points=64)
    out2, req2 = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out), **sub)
    sp = W.subset_points(pts, np.arange(1000, 1064))
    o2, oreq2 = oracle.run_points(m, traces, sp, per_request=True)
    compare_points(out2, o2, "c3 sub-range")
    compare_requests(req2, oreq2, "c3 sub-range")


def test_full_c4_points(S, oracle):
    m, traces, pts = W.make_config("c4")
    t0 = time.time()
    o_out, _ = oracle.run_points(m, traces, pts)
    say("c4: oracle %.1fs, %d preemptions" % (time.time() - t0, int(o_out["n_preempt"].sum())))
    out, _ = gpu_run(S, m, traces, pts, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "c4")


@pytest.mark.parametrize("name", ["c6x", "c7x", "c8x", "c4u"])
def test_gpu_filling_sweeps_all_points(S, oracle, name):
    """The policy, swap and disaggregation studies at a size that fills the
    GPU (at least 8192 simulation units), and c4 with one trace per point:
    every point's counters, sums, percentiles and request digest."""
    m, traces, pts = W.make_config(name)
    t0 = time.time()
    o_out, _ = oracle.run_points(m, traces, pts)
    say("%s: oracle on all %d points %.1fs" % (name, len(pts["peak_flops"]), time.time() - t0))
    out, _ = gpu_run(S, m, traces, pts, iter_cap=cap_from(o_out))
    compare_points(out, o_out, name)
    assert (out["status"] == 0).all()


def test_c5_all_points(S, oracle):
    """The full 65536-point x 10000-request c5 sweep, launched as the
    benchmark launches it: every point's counters, sums, percentiles and
    request digest against the oracle."""
    m, traces, pts = W.make_config("c5")
    n_pts = len(pts["peak_flops"])
    t0 = time.time()
    o_out, _ = oracle.run_points(m, traces, pts)
    say("c5: oracle on all %d points %.1fs (%d threads)" % (n_pts, time.time() - t0,
                                                          oracle.default_threads()))
    out, _ = gpu_run(S, m, traces, pts, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "c5")
    assert (out["status"] == 0).all()
    # properties that hold at any size
    n = len(traces[0]["arrival_ns"])
    assert (out["n_done"] + out["n_rejected"] == n).all()
    tr_o = np.array([int(t["output_len"].sum()) for t in traces])
    assert (out["decode_tokens"] == tr_o[pts["trace_id"]]).all()
    tr_p = np.array([int(t["prompt_len"].sum()) for t in traces])
    assert (out["prefill_tokens"] >= tr_p[pts["trace_id"]]).all()
    assert (out["peak_used_blocks"] <= out["num_blocks"]).all()


def test_c5_full_size_per_request(S, oracle):
    """512 seeded c5 points at the full 10000 requests: every request record."""
    m, traces, pts = W.make_config("c5")
    idx = np.sort(np.random.default_rng(5).choice(len(pts["peak_flops"]), 512, replace=False))
    sub = W.subset_points(pts, idx)
    o_out, o_req = oracle.run_points(m, traces, sub, per_request=True)
    out, req = gpu_run(S, m, traces, sub, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "c5 per request")
    compare_requests(req, o_req, "c5 per request")


def test_rerun_same_handle_other_stream(S, oracle):
    """One handle run twice, the second time on another stream: both runs
    equal the oracle (the benchmark times re-runs of one handle)."""
    import torch
    m, traces, pts = W.make_config("c2")
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    sw = S.Sweep(m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    try:
        sw.run(torch.cuda.current_stream())
        a, ra = sw.results()
        compare_points(a, o_out, "first run")
        compare_requests(ra, o_req, "first run")
        other = torch.cuda.Stream()
        sw.run(torch.cuda.current_stream())
        sw.run(other)  # ordered after the run before it, on the device
        b, rb = sw.results()
        compare_points(b, o_out, "re-run")
        compare_requests(rb, o_req, "re-run")
        assert a.tobytes() == b.tobytes() and ra.tobytes() == rb.tobytes()
        sim_ms, stats_ms = sw.timing()
        assert sim_ms > 0 and stats_ms >= 0
    finally:
        sw.close()


def test_call_order_errors(S):
    """results / timing before the first run, and request records asked of a
    handle created without them, are TS_ERR_STATE."""
    import ctypes as C
    m, traces, pts = W.make_config("c1")
    sw = S.Sweep(m, traces, pts, iter_cap=100_000)
    try:
        for call in (sw.results, sw.timing, sw.kernel_timing):
            with pytest.raises(S.SweepError) as ei:
                call()
            assert ei.value.rc == S.TS_ERR_STATE
        sw.run()
        out, req = sw.results()
        assert req is None and out["n_done"][0] == 64
        pbuf = np.zeros(1, dtype=S.POINT_DTYPE)
        rbuf = np.zeros((1, sw.max_n), dtype=S.REQ_DTYPE)
        rc = S.lib().ts_sweep_results(sw._h, C.c_void_p(pbuf.ctypes.data),
                                      C.c_void_p(rbuf.ctypes.data))
        assert rc == S.TS_ERR_STATE
    finally:
        sw.close()


def test_device_memory_shortage_is_oom(S):
    """A sweep whose buffers exceed the device's memory fails with
    TS_ERR_OOM at create, before any allocation; the library stays usable."""
    m = W.MODELS["llama2-7b"]
    n = 1_000_000
    tr = {"arrival_ns": np.arange(n, dtype=np.int64), "prompt_len": np.full(n, 8, np.int32),
          "output_len": np.full(n, 8, np.int32)}
    k = 20_000  # latency arrays alone: 20000 points x 1e6 requests x 16 B = 320 GB
    pts = {"peak_flops": np.full(k, 312e12), "mem_bw": np.full(k, 2e12),
           "capacity_bytes": np.full(k, 80_000_000_000, np.int64),
           "mem_util_permille": np.full(k, 900, np.int32),
           "block_size": np.full(k, 16, np.int32), "max_batch": np.full(k, 64, np.int32),
           "chunk_size": np.zeros(k, np.int32), "trace_id": np.zeros(k, np.int32)}
    with pytest.raises(S.SweepError) as ei:
        S.Sweep(m, [tr], pts, iter_cap=1)
    assert ei.value.rc == S.TS_ERR_OOM
    assert "device memory" in S.lib().ts_status_str(S.TS_ERR_OOM).decode()
    m1, t1, p1 = W.make_config("c1")
    out, _ = gpu_run(S, m1, t1, p1, iter_cap=100_000)
    assert out["n_done"][0] == 64


def test_watchdog_path_per_request(S, oracle):
    """With the wall-clock watchdog on, steady stretches stop every 256
    iterations for its clock check: the same results, request by request."""
    m, traces, pts = W.make_config("c2")
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out),
                       point_time_limit_ms=60_000)
    compare_points(out, o_out, "watchdog")
    compare_requests(req, o_req, "watchdog")


@pytest.mark.parametrize("name,nreq", [("c5", 2000), ("c4", 1000), ("c3", 1000)])
def test_sweep_subsets_per_request(S, oracle, name, nreq):
    """2048 seeded points of a large sweep at fewer requests per trace,
    every point and every request against the oracle (both chunk classes,
    chunked prefill, heavy preemption)."""
    m, traces, pts = W.make_config(name, n_requests=nreq)
    n = len(pts["peak_flops"])
    idx = np.sort(np.random.default_rng(7).choice(n, size=min(2048, n), replace=False))
    pts = W.subset_points(pts, idx)
    t0 = time.time()
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    say("%s subset: oracle %.1fs, preemptions %d" % (name, time.time() - t0,
                                                     int(o_out["n_preempt"].sum())))
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, name)
    compare_requests(req, o_req, name)
    assert len(set(pts["max_batch"].tolist())) > 1 or name == "c4"


@pytest.mark.parametrize("seed,takeover", [(3, True), (4, True), (5, True), (6, True),
                                           (3, False), (4, False)])
def test_hand_over_records_under_memory_pressure(S, oracle, seed, takeover):
    """Simple points of every width up to 256 slots under bursts of up to
    260 simultaneous arrivals and small KV budgets: points continue in the
    wider launches from their hand-over records with running requests,
    reserved blocks and preempted requests waiting (or start over when a
    window had already admitted), with and without the 64-slot launch's
    take-over of its own handed points.  Every request against the oracle;
    the launches' iteration counts add up to the oracle's."""
    m = {"n_layers": 2, "d_model": 64, "n_heads": 4, "n_kv_heads": 2, "ffn_dim": 128,
         "ffn_gated": 1, "vocab": 100, "w_bytes": 2, "kv_bytes": 2, "weights_in_capacity": 0}
    rng = np.random.default_rng(seed)
    traces = []
    for _ in range(6):
        groups = rng.integers(1, 260, size=8)
        arr = np.sort(np.concatenate([np.full(g, int(rng.integers(0, 2_000_000_000)))
                                      for g in groups]))[:int(rng.integers(150, 400))]
        n = len(arr)
        traces.append({"arrival_ns": arr.astype(np.int64),
                       "prompt_len": rng.integers(1, 300, n).astype(np.int32),
                       "output_len": rng.integers(1, 120, n).astype(np.int32)})
    k = 60
    kv_tok = 2 * 2 * (64 // 4 * 2) * 2
    pts = {"peak_flops": rng.choice([1e12, 5e12, 2e13], k),
           "mem_bw": rng.choice([1e11, 5e11, 2e12], k),
           "capacity_bytes": (rng.integers(200, 6000, k) * kv_tok * 16).astype(np.int64),
           "mem_util_permille": np.full(k, 1000, np.int32),
           "block_size": rng.choice([1, 4, 16], k).astype(np.int32),
           "max_batch": rng.choice([64, 65, 100, 128, 129, 200, 256], k).astype(np.int32),
           "trace_id": rng.integers(0, len(traces), k).astype(np.int32)}
    ch = rng.choice([0, 256, 512, 1024], k)
    pts["chunk_size"] = np.where(ch == 0, 0, np.maximum(ch, pts["max_batch"])).astype(np.int32)
    # only points that reject nothing (the hand-over needs every point simple)
    o_all, _ = oracle.run_points(m, traces, pts)
    pts = W.subset_points(pts, np.nonzero(o_all["n_rejected"] == 0)[0])
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    sw = S.Sweep(m, traces, pts, per_request=True, iter_cap=cap_from(o_out), takeover=takeover)
    try:
        sw.run()
        out, req = sw.results()
        work = sw.kernel_work()
    finally:
        sw.close()
    compare_points(out, o_out, "hand-over records")
    compare_requests(req, o_req, "hand-over records")
    assert work[2] > 0
    if not takeover:
        assert work[1] > 0
    assert int(o_out["n_preempt"].sum()) > 50
    assert sum(work) == int(o_out["n_iters"].sum())


@pytest.mark.parametrize("seed", [11, 12])
def test_blocks_through_simultaneous_finishes(S, oracle, seed):
    """Simple points whose decodes finish while a long head prefill runs:
    groups of requests with equal outputs admitted together finish in the
    same iteration, short prompts ride behind long chunked ones, and tight
    KV budgets with block sizes 1 to 16 make iterations run short of blocks
    inside a block of iterations.  Every request against the oracle."""
    m = {"n_layers": 2, "d_model": 64, "n_heads": 4, "n_kv_heads": 2, "ffn_dim": 128,
         "ffn_gated": 1, "vocab": 100, "w_bytes": 2, "kv_bytes": 2, "weights_in_capacity": 0}
    rng = np.random.default_rng(seed)
    traces = []
    for _ in range(4):
        n = int(rng.integers(150, 300))
        arr = np.sort(rng.integers(0, 400_000_000, n)).astype(np.int64)
        arr[: n // 3] = arr[0]  # a burst admitted together
        prompt = np.where(rng.random(n) < 0.3, rng.integers(600, 3000, n),
                          rng.integers(1, 60, n)).astype(np.int32)
        output = rng.choice([8, 16, 17, 40], n).astype(np.int32)  # equal outputs finish together
        traces.append({"arrival_ns": arr, "prompt_len": prompt, "output_len": output})
    k = 48
    kv_tok = 2 * 2 * (64 // 4 * 2) * 2
    pts = {"peak_flops": rng.choice([1e12, 5e12], k), "mem_bw": rng.choice([1e11, 1e12], k),
           "capacity_bytes": (rng.integers(3200, 20000, k) * kv_tok).astype(np.int64),
           "mem_util_permille": np.full(k, 1000, np.int32),
           "block_size": rng.choice([1, 2, 4, 16], k).astype(np.int32),
           "max_batch": rng.choice([16, 64, 100, 128], k).astype(np.int32),
           "trace_id": rng.integers(0, len(traces), k).astype(np.int32)}
    pts["chunk_size"] = np.maximum(rng.choice([64, 128, 256], k), pts["max_batch"]).astype(np.int32)
    o_all, _ = oracle.run_points(m, traces, pts)
    pts = W.subset_points(pts, np.nonzero(o_all["n_rejected"] == 0)[0])  # simple points only
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "simultaneous finishes")
    compare_requests(req, o_req, "simultaneous finishes")
    assert int(o_out["n_done"].sum()) > 5000


def test_percentiles_when_many_latencies_are_equal(S, oracle):
    """Requests served one at a time with equal lengths have equal latencies:
    far more of them share a latency bucket than the statistics kernel keeps
    in LDS, so those percentiles come from radix passes over the whole
    latency array; one point has a few longer requests, so its p99 lies in
    another bucket."""
    m = W.MODELS["llama2-7b"]
    n = 1500
    rng = np.random.default_rng(7)
    gaps = np.arange(n, dtype=np.int64) * 10_000_000_000
    same = {"arrival_ns": gaps, "prompt_len": np.full(n, 100, np.int32),
            "output_len": np.full(n, 50, np.int32)}
    out_len = np.full(n, 50, np.int32)
    out_len[rng.choice(n, 40, replace=False)] = 400
    mixed = {"arrival_ns": gaps, "prompt_len": np.full(n, 100, np.int32), "output_len": out_len}
    pts = {"peak_flops": np.full(2, 312e12), "mem_bw": np.full(2, 2e12),
           "capacity_bytes": np.full(2, 80_000_000_000, np.int64),
           "mem_util_permille": np.full(2, 900, np.int32), "block_size": np.full(2, 16, np.int32),
           "max_batch": np.full(2, 64, np.int32), "chunk_size": np.zeros(2, np.int32),
           "trace_id": np.array([0, 1], np.int32)}
    traces = [same, mixed]
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "equal latencies")
    compare_requests(req, o_req, "equal latencies")
    assert out["p50_e2e_ns"][0] == out["p99_e2e_ns"][0]
    assert out["p99_e2e_ns"][1] > out["p50_e2e_ns"][1]


def test_determinism_and_point_order(S):
    m, traces, pts = W.make_config("c3", n_requests=300)
    n = len(pts["peak_flops"])
    a, _ = gpu_run(S, m, traces, pts, iter_cap=1_000_000)
    b, _ = gpu_run(S, m, traces, pts, iter_cap=1_000_000)
    assert a.tobytes() == b.tobytes()
    perm = np.random.default_rng(1).permutation(n)
    c, _ = gpu_run(S, m, traces, W.subset_points(pts, perm), iter_cap=1_000_000)
    assert c.tobytes() == a[perm].tobytes()


def test_edge_cases(S, oracle):
    m = W.MODELS["llama2-7b"]
    empty = {"arrival_ns": np.zeros(0, np.int64), "prompt_len": np.zeros(0, np.int32),
             "output_len": np.zeros(0, np.int32)}
    burst = {"arrival_ns": np.zeros(300, np.int64),
             "prompt_len": np.full(300, 64, np.int32), "output_len": np.full(300, 40, np.int32)}
    huge = {"arrival_ns": np.array([0, 5, 9], np.int64),
            "prompt_len": np.array([10, 200000, 10], np.int32),
            "output_len": np.array([3, 3, 3], np.int32)}
    traces = [empty, burst, huge]
    rows = [
        (312e12, 2e12, 80_000_000_000, 900, 16, 32, 0, 0),     # empty trace
        (312e12, 2e12, 80_000_000_000, 900, 16, 256, 0, 1),    # 300 at once, M = 256
        (312e12, 2e12, 80_000_000_000, 900, 16, 256, 256, 1),  # chunk = M
        (312e12, 2e12, 14_000_000_000, 1000, 16, 256, 0, 1),   # tight memory: preemption
        (312e12, 2e12, 10_000_000_000, 900, 16, 8, 0, 1),      # weights > capacity: NO_KV
        (312e12, 2e12, 20_000_000_000, 1000, 16, 8, 0, 2),     # one request rejected
        (312e12, 2e12, 80_000_000_000, 900, 1, 130, 512, 1),   # block 1, two chunks
    ]
    keys = ("peak_flops", "mem_bw", "capacity_bytes", "mem_util_permille", "block_size",
            "max_batch", "chunk_size", "trace_id")
    pts = {k: np.array([r[i] for r in rows]) for i, k in enumerate(keys)}
    pts = {k: (v.astype(np.float64) if k in ("peak_flops", "mem_bw", "swap_bw") else
               v.astype(np.int64) if k == "capacity_bytes" else v.astype(np.int32))
           for k, v in pts.items()}
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    assert o_out["status"][4] == 1 and o_out["n_rejected"][5] == 1 and o_out["n_preempt"][3] > 0
    out, req = gpu_run(S, m, traces, pts, per_request=True, iter_cap=cap_from(o_out))
    compare_points(out, o_out, "edge")
    compare_requests(req, o_req, "edge")
    # iteration cap: stops early, identical partial state
    o_cap, o_rq = oracle.run_points(m, traces, pts, per_request=True, iter_cap=37)
    g_cap, g_rq = gpu_run(S, m, traces, pts, per_request=True, iter_cap=37)
    compare_points(g_cap, o_cap, "iter cap")
    compare_requests(g_rq, o_rq, "iter cap")
    assert (g_cap["status"][[1, 2, 3, 6]] == 2).all()


@pytest.mark.parametrize("takeover", [True, False])
def test_hand_over_to_wider_kernels(S, oracle, takeover):
    """Simple one-worker points with room for more than 64 running requests
    first run in the 64-slot kernel; those that need more slots (bursts of
    300 arrivals) are handed on with 128 slots (continued by the 64-slot
    launch itself once none of its own points is left, or else by the
    128-slot launch) and from there to the 256-slot launch; without the
    take-over the 128-slot launch continues every one.  Every request
    against the oracle, and the launches' completed iterations add up to the
    oracle's."""
    m = W.MODELS["llama2-7b"]
    rng = np.random.default_rng(3)
    burst = {"arrival_ns": np.zeros(300, np.int64),
             "prompt_len": rng.integers(16, 200, 300).astype(np.int32),
             "output_len": rng.integers(5, 60, 300).astype(np.int32)}
    n = 400
    spread = {"arrival_ns": np.sort(rng.integers(0, 3_000_000_000, n)).astype(np.int64),
              "prompt_len": rng.integers(16, 2000, n).astype(np.int32),
              "output_len": rng.integers(5, 300, n).astype(np.int32)}
    rows = [(256, 0, 0), (100, 0, 0), (64, 0, 0), (256, 512, 0), (130, 256, 1), (256, 0, 1),
            (80, 0, 1), (256, 1024, 1)]
    k = len(rows)
    pts = {"peak_flops": np.full(k, 312e12), "mem_bw": np.full(k, 2e12),
           "capacity_bytes": np.full(k, 80_000_000_000, np.int64),
           "mem_util_permille": np.full(k, 900, np.int32), "block_size": np.full(k, 16, np.int32),
           "max_batch": np.array([r[0] for r in rows], np.int32),
           "chunk_size": np.array([r[1] for r in rows], np.int32),
           "trace_id": np.array([r[2] for r in rows], np.int32)}
    traces = [burst, spread]
    o_out, o_req = oracle.run_points(m, traces, pts, per_request=True)
    sw = S.Sweep(m, traces, pts, per_request=True, iter_cap=cap_from(o_out), takeover=takeover)
    try:
        sw.run()
        out, req = sw.results()
        work = sw.kernel_work()
        per_launch = [kt[1] for kt in sw.kernel_timing()]
    finally:
        sw.close()
    compare_points(out, o_out, "hand-over")
    compare_requests(req, o_req, "hand-over")
    assert per_launch[0] == k  # the 64-slot launch takes every point
    assert work[2] > 0  # bursts were handed on twice (64 -> 128 -> 256 slots)
    if not takeover:
        assert work[1] > 0  # the 128-slot launch continued them
    assert sum(work) == int(o_out["n_iters"].sum())
