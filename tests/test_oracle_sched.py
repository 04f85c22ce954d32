"""Pins for the oracle's scheduler, clock and statistics.

Hand-traced schedules, closed forms that follow from the paper's
description of continuous batching (Sec. II-B, Sec. IV-A), the under-load
latency shape of the simulator comparison table (Sec. III-D), invariants
checked after every iteration, and the statistics definitions checked
against library routines.
"""
import json
import os

import numpy as np
import pytest

from paper_2503_08415_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")
INF = 1e300


def _trace(reqs):
    a = np.array([r[0] for r in reqs], dtype=np.int64)
    p = np.array([r[1] for r in reqs], dtype=np.int32)
    o = np.array([r[2] for r in reqs], dtype=np.int32)
    return {"arrival_ns": a, "prompt_len": p, "output_len": o}


def _hand_cases():
    with open(os.path.join(GOLD, "hand_traces.json")) as f:
        g = json.load(f)
    return g["model"], g["cases"]


HAND_MODEL, HAND_CASES = _hand_cases()


def hand_point(case):
    nb, b = case["num_blocks"], case["block_size"]
    cap = nb * b * 16 if nb > 0 else 1   # the toy model stores 16 B of KV per token
    pt = dict(peak_flops=INF, mem_bw=INF, capacity_bytes=cap, mem_util_permille=1000,
              block_size=b, max_batch=case["max_batch"], chunk_size=case["chunk_size"],
              policy=case.get("policy", 0),
              admit_mem_permille=case.get("admit_mem_permille", 0),
              swap_bw=case.get("swap_bw", 0.0), swap_overlap=case.get("swap_overlap", 0))
    if case.get("n_prefill", 0) > 0:  # disaggregated: prefill devices as fast, own memory
        pt.update(n_prefill=case["n_prefill"], n_decode=case["n_decode"], p_peak_flops=INF,
                  p_mem_bw=INF, p_capacity_bytes=max(1, case["prefill_blocks"] * b * 16),
                  kv_link_bw=case["kv_link_bw"])
    return pt


@pytest.mark.parametrize("case", HAND_CASES, ids=[c["name"] for c in HAND_CASES])
def test_hand_traced_schedules(oracle, case):
    log_cap = 0 if case.get("n_prefill", 0) > 0 else 1000
    out, req, log, viol = oracle.simulate_point(HAND_MODEL, _trace(case["requests"]),
                                                hand_point(case), log_cap=log_cap)
    assert viol == 0
    got = [[int(r["admit_ns"]), int(r["first_token_ns"]), int(r["finish_ns"]),
            int(r["max_gap_ns"]), int(r["n_preempt"]), int(r["status"])] for r in req]
    assert got == case["expect_req"]
    for k, v in case["expect_point"].items():
        assert out[k] == v, k
    assert out["num_blocks"] == case["num_blocks"]


C1_MODEL = W.MODELS["llama2-7b"]
A100 = dict(peak_flops=312e12, mem_bw=2.0e12, capacity_bytes=80_000_000_000,
            mem_util_permille=900, block_size=16, max_batch=32, chunk_size=0)


def _costs(oracle, point):
    d = oracle.derive(C1_MODEL, point)
    return lambda batch: oracle.iter_ns(C1_MODEL, d["inv_flops_ns"], d["inv_bw_ns"], batch)


def test_single_request_closed_form(oracle):
    """TTFT = queueing + prefill cost; then exactly output_len decodes."""
    cost = _costs(oracle, A100)
    for arr, p, o in [(0, 1, 1), (5_000, 700, 9), (123_456_789, 3000, 40)]:
        out, req, log, viol = oracle.simulate_point(C1_MODEL, _trace([(arr, p, o)]), A100,
                                                    log_cap=100)
        assert viol == 0
        r = req[0]
        assert r["admit_ns"] == arr
        assert r["first_token_ns"] == arr + cost([(p, 0, 1, 1)])
        dec = [cost([(1, p + j, 0, 0)]) for j in range(o)]
        assert r["finish_ns"] == r["first_token_ns"] + sum(dec)
        assert r["max_gap_ns"] == max(dec)
        assert out["n_iters"] == 1 + o and out["decode_tokens"] == o
        assert out["prefill_tokens"] == p and out["n_preempt"] == 0


def test_queueing_adds_to_ttft(oracle):
    """With max batch 1 the second request's TTFT = first's finish - arrival
    + its own prefill."""
    pt = dict(A100, max_batch=1)
    cost = _costs(oracle, pt)
    out, req, _, viol = oracle.simulate_point(C1_MODEL, _trace([(0, 300, 5), (0, 200, 3)]), pt)
    assert viol == 0
    assert req[1]["admit_ns"] == req[0]["finish_ns"]
    assert req[1]["first_token_ns"] == req[0]["finish_ns"] + cost([(200, 0, 1, 1)])


def test_synchronised_batch(oracle):
    """N identical requests at t=0 with room for all: one prefill iteration
    over N*p tokens, then o decodes of batch N (the textbook static batch)."""
    cost = _costs(oracle, A100)
    n, p, o = 8, 128, 20
    out, req, _, viol = oracle.simulate_point(C1_MODEL, _trace([(0, p, o)] * n), A100)
    assert viol == 0
    first = cost([(p, 0, 1, 1)] * n)
    assert (req["first_token_ns"] == first).all()
    fin = first + sum(cost([(1, p + j, 0, 0)] * n) for j in range(o))
    assert (req["finish_ns"] == fin).all()
    assert out["n_iters"] == 1 + o


def test_under_load_latency_shape(oracle):
    """Table II (Sec. III-D): at a fixed 40 requests/s with 10 output tokens the
    makespan grows as (N-1)/40 s plus about one request's latency (the
    paper's TokenSim column: 2.592 .. 12.593 s for N = 100 .. 500)."""
    pt = dict(A100, max_batch=256)
    cost = _costs(oracle, pt)
    p = 512  # a prompt length at which 40 requests/s is below saturation
    single = cost([(p, 0, 1, 1)]) + sum(cost([(1, p + j, 0, 0)]) for j in range(10))
    tails = []
    for n in (100, 200, 300, 400, 500):
        reqs = [(i * 25_000_000, p, 10) for i in range(n)]
        out, req, _, viol = oracle.simulate_point(C1_MODEL, _trace(reqs), pt)
        assert viol == 0 and out["n_done"] == n
        tails.append(int(req["finish_ns"].max()) - (n - 1) * 25_000_000)
    assert max(tails) - min(tails) < 5_000_000                 # constant tail
    assert single <= min(tails) < 1.5 * single                 # about one request
    assert 0.08e9 < np.mean(tails) < 0.15e9                    # paper: 0.112 .. 0.120 s


def _shrunk(name, n_req, n_pts, seed):
    m, traces, pts = W.make_config(name, n_requests=n_req)
    rng = np.random.default_rng(seed)
    idx = rng.choice(len(pts["peak_flops"]), size=n_pts, replace=False)
    return m, traces, W.subset_points(pts, idx)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_invariants_every_iteration(oracle, name):
    m, traces, pts = _shrunk(name, 150 if name != "c1" else 64, 1 if name == "c1" else 6, 3)
    # memory pressure: scale capacity down so preemption triggers
    for i in range(len(pts["peak_flops"])):
        p = {k: v[i] for k, v in pts.items()}
        for shrink in (1, 4):
            q = dict(p)
            if not m["weights_in_capacity"]:
                q["capacity_bytes"] = max(1, int(p["capacity_bytes"]) // (20 * shrink))
            out, req, _, viol = oracle.simulate_point(m, traces[int(p["trace_id"])], q)
            assert viol == 0
            if out["status"] == 0:
                done = req["status"] == 1
                assert out["n_done"] + out["n_rejected"] == len(req)
                o = traces[int(p["trace_id"])]["output_len"]
                assert out["decode_tokens"] == int(o[done].sum())


def test_preemption_triggers_under_pressure(oracle):
    m, traces, pts = _shrunk("c4", 400, 4, 11)
    total = 0
    for i in range(4):
        p = {k: v[i] for k, v in pts.items()}
        p["capacity_bytes"] = int(p["capacity_bytes"]) // 8
        out, req, _, viol = oracle.simulate_point(m, traces[int(p["trace_id"])], p)
        assert viol == 0
        total += out["n_preempt"]
        pr = traces[int(p["trace_id"])]["prompt_len"]
        done = req["status"] == 1
        assert out["prefill_tokens"] >= int(pr[done].sum())
        if out["n_preempt"] > 0:
            assert out["prefill_tokens"] > int(pr[done].sum())
        assert int(req["n_preempt"].sum()) == out["n_preempt"]
    assert total > 0


def test_statistics_definitions(oracle):
    m, traces, pts = _shrunk("c2", 400, 3, 5)
    for i in range(3):
        p = {k: v[i] for k, v in pts.items()}
        tr = traces[int(p["trace_id"])]
        out, req, _, _ = oracle.simulate_point(m, tr, p, slo_ttft_ns=2_000_000_000,
                                               slo_tpot_ns=60_000_000)
        done = req["status"] == 1
        arr = tr["arrival_ns"][done]
        e2e = req["finish_ns"][done] - arr
        ttft = req["first_token_ns"][done] - arr
        # nearest rank = numpy's inverted-CDF percentile
        for pct, key in ((50, "p50_e2e_ns"), (90, "p90_e2e_ns"), (99, "p99_e2e_ns")):
            assert out[key] == int(np.percentile(e2e, pct, method="inverted_cdf"))
        for pct, key in ((50, "p50_ttft_ns"), (99, "p99_ttft_ns")):
            assert out[key] == int(np.percentile(ttft, pct, method="inverted_cdf"))
        assert out["sum_e2e_ns"] == int(e2e.sum()) and out["sum_ttft_ns"] == int(ttft.sum())
        assert out["max_e2e_ns"] == int(e2e.max())
        assert out["sum_tpot_num_ns"] == int((req["finish_ns"][done] - req["first_token_ns"][done]).sum())
        ok = (ttft <= 2_000_000_000) & (req["max_gap_ns"][done] <= 60_000_000)
        assert out["slo_ok"] == int(ok.sum())
        assert out["slo_tpot_ok"] == int((req["max_gap_ns"][done] <= 60_000_000).sum())
        assert out["slo_ok"] <= out["slo_tpot_ok"] <= out["n_done"]
        # a TTFT objective at the median separates the two counts
        tight = int(np.median(ttft))
        out2, _, _, _ = oracle.simulate_point(m, tr, p, slo_ttft_ns=tight,
                                              slo_tpot_ns=60_000_000)
        ok2 = (ttft <= tight) & (req["max_gap_ns"][done] <= 60_000_000)
        assert out2["slo_ok"] == int(ok2.sum()) and out2["slo_tpot_ok"] == out["slo_tpot_ok"]
        assert out2["slo_ok"] < out2["slo_tpot_ok"]
        assert out["last_finish_ns"] == int(req["finish_ns"][done].max())
        assert out["first_arrival_ns"] == int(tr["arrival_ns"][0])


def _fmix64(k):
    M = (1 << 64) - 1
    k ^= k >> 33
    k = (k * 0xff51afd7ed558ccd) & M
    k ^= k >> 33
    k = (k * 0xc4ceb9fe1a85ec53) & M
    k ^= k >> 33
    return k


def test_digest_definition(oracle):
    M = (1 << 64) - 1
    m, traces, pts = _shrunk("c3", 300, 2, 9)
    for i in range(2):
        p = {k: v[i] for k, v in pts.items()}
        out, req, _, _ = oracle.simulate_point(m, traces[int(p["trace_id"])], p)
        acc = 0
        for idx, r in enumerate(req):
            if r["status"] == 0:
                continue
            tail = ((int(r["n_preempt"]) & 0xffffffff) << 32) | int(r["status"])
            fields = (idx, int(r["admit_ns"]), int(r["first_token_ns"]), int(r["finish_ns"]),
                      int(r["max_gap_ns"]), tail)
            mult = (0x9e3779b97f4a7c15, 0xbf58476d1ce4e5b9, 0x94d049bb133111eb,
                    0xd6e8feb86659fd93, 0xa0761d6478bd642f, 0xe7037ed1a0b428db)
            h = sum((v & M) * k for v, k in zip(fields, mult)) & M
            acc = (acc + _fmix64(h)) & M
        assert int(out["digest"]) == acc


def test_empty_trace_and_iteration_cap(oracle):
    empty = {"arrival_ns": np.zeros(0, np.int64), "prompt_len": np.zeros(0, np.int32),
             "output_len": np.zeros(0, np.int32)}
    out, req, _, _ = oracle.simulate_point(C1_MODEL, empty, A100)
    assert out["status"] == 0 and out["n_iters"] == 0 and out["first_arrival_ns"] == -1
    assert out["p50_e2e_ns"] == -1 and out["max_e2e_ns"] == -1
    tr = _trace([(0, 50, 30), (10, 20, 30)])
    out, req, _, _ = oracle.simulate_point(C1_MODEL, tr, A100, iter_cap=7)
    assert out["status"] == 2 and out["n_iters"] == 7
    assert (req["status"] == 0).all() and (req["admit_ns"] == -1).all()


def test_bad_arguments_rejected(oracle):
    tr = _trace([(0, 5, 5)])
    for bad in (dict(A100, chunk_size=8), dict(A100, block_size=0), dict(A100, policy=3),
                dict(A100, policy=-1), dict(A100, policy=1, chunk_size=256),
                dict(A100, admit_mem_permille=1001), dict(A100, admit_mem_permille=-1),
                dict(A100, peak_flops=float("inf")), dict(A100, mem_util_permille=0)):
        with pytest.raises(oracle.OracleError):
            oracle.simulate_point(C1_MODEL, tr, bad)
    with pytest.raises(oracle.OracleError):
        oracle.simulate_point(C1_MODEL, _trace([(10, 5, 5), (0, 5, 5)]), A100)


def test_thread_count_does_not_change_results(oracle):
    m, traces, pts = _shrunk("c3", 300, 16, 2)
    a, ra = oracle.run_points(m, traces, pts, per_request=True, n_threads=1)
    b, rb = oracle.run_points(m, traces, pts, per_request=True, n_threads=8)
    assert a.tobytes() == b.tobytes() and ra.tobytes() == rb.tobytes()
