"""Pins for the oracle's disaggregated design points (prefill and decode on
separate devices, Sec. II-B; breakpoints and a global scheduler, Sec. III-A;
KV transfers priced by the communication model, Sec. III-B).

The oracle runs such a point in stages: every prefill device on its own,
then every decode device on the requests whose KV has reached it.  The
brute force below is a different formulation: one global event loop over
all devices that always runs the device whose next iteration starts first,
moving each request to its decode device when its transfer ends.  Requests
are dicts and every block count is recomputed from token counts.  Iteration
costs come from the oracle's cost function (pinned separately).
"""
import math
import random

import numpy as np
import pytest

TOY = {"n_layers": 1, "d_model": 8, "n_heads": 2, "n_kv_heads": 1, "ffn_dim": 16,
       "ffn_gated": 1, "vocab": 10, "w_bytes": 2, "kv_bytes": 2, "weights_in_capacity": 0}
KV_TOKEN = 2 * TOY["n_layers"] * (TOY["n_kv_heads"] * TOY["d_model"] // TOY["n_heads"]) * \
    TOY["kv_bytes"]  # 16 bytes of K and V per token


def blocks(tokens, b):
    return -(-tokens // b)


class Device:
    """One simulated device: its requests, its clock and its counters."""

    def __init__(self, prefill, NB, b, M, K, cost, permille=0, swap_bw=0.0, overlap=0):
        self.prefill = prefill
        self.NB, self.b, self.M, self.K, self.cost = NB, b, M, K, cost
        self.reserve = NB - (NB * permille // 1000 if permille else NB)
        self.inv_link = 1e9 / swap_bw if swap_bw > 0 else 0.0
        self.swap = swap_bw > 0
        self.overlap = overlap
        self.reqs = []
        self.clock = 0
        self.seq = 0
        self.iters = self.n_pre = self.pre_tok = self.dec_tok = self.peak = 0
        self.ubns = 0.0

    def held(self, r):
        return blocks(max(r["ctx"], r["tgt"]), self.b)

    def running(self):
        return sorted([r for r in self.reqs if r["ph"] == "run"], key=lambda r: r["seq"])

    def waiting(self):
        return sorted([r for r in self.reqs if r["ph"] == "wait"], key=lambda r: (r["at"], r["gid"]))

    def free(self):
        return self.NB - sum(self.held(r) for r in self.running())

    def next_start(self):
        new = [r["at"] for r in self.reqs if r["ph"] == "new"]
        if self.running() or self.waiting() or any(a <= self.clock for a in new):
            return self.clock
        return min(new) if new else None

    def iterate(self, t):
        """One iteration starting at t; returns the requests whose prefill
        completed on a prefill device, in slot order."""
        b = self.b
        for r in self.reqs:
            if r["ph"] == "new" and r["at"] <= t:
                r["ph"] = "wait"
        grow, moved, preempted = set(), 0, False
        for r in self.running():
            if r["ph"] != "run" or not (r["ctx"] >= r["tgt"] and r["ctx"] % b == 0):
                continue
            while self.free() - len(grow) == 0:
                v = max(self.running(), key=lambda x: x["seq"])
                if self.swap:
                    moved += self.held(v)
                    v.update(ph="wait", sw=True, npre=v["npre"] + 1)
                else:
                    v.update(ph="wait", ctx=0, tgt=v["p"] + v["gd"], npre=v["npre"] + 1)
                grow.discard(v["gid"])
                self.n_pre += 1
                preempted = True
                if v is r:
                    break
            if r["ph"] == "run":
                grow.add(r["gid"])
        budget = None if self.K == 0 else \
            self.K - sum(1 for r in self.running() if r["ctx"] >= r["tgt"])
        q = {}
        for r in self.running():
            if r["ctx"] < r["tgt"]:
                left = r["tgt"] - r["ctx"]
                q[r["gid"]] = left if budget is None else min(left, budget)
                if budget is not None:
                    budget -= q[r["gid"]]
        idle = set()
        if not preempted:
            for h in self.waiting():
                if len(self.running()) >= self.M:
                    break
                if not h["sw"] and budget is not None and budget <= 0:
                    break
                if h["sw"]:
                    need = self.held(h)
                elif h["ctx"] >= h["tgt"]:  # arrived with its KV: holds the next token too
                    need = blocks(h["ctx"] + 1, b)
                else:
                    need = blocks(h["tgt"], b)
                room = self.free() - len(grow) - (self.reserve if h["fresh"] else 0)
                if need > room:
                    break
                self.seq += 1
                h.update(ph="run", seq=self.seq, fresh=False)
                if h["admit"] < 0:
                    h["admit"] = t
                if h["sw"]:
                    moved += need
                    h["sw"] = False
                    idle.add(h["gid"])
                elif h["ctx"] >= h["tgt"]:
                    if need > self.held(h):
                        grow.add(h["gid"])
                    if budget is not None:
                        budget -= 1
                else:
                    q[h["gid"]] = h["tgt"] if budget is None else min(h["tgt"], budget)
                    if budget is not None:
                        budget -= q[h["gid"]]
        run = self.running()
        used = self.NB - self.free() + len(grow)
        batch = []
        for r in run:
            if r["gid"] in idle:
                continue
            if r["ctx"] >= r["tgt"]:
                batch.append((1, r["ctx"], 0, 0))
            elif q.get(r["gid"], 0) > 0:
                comp = int(r["ctx"] + q[r["gid"]] == r["tgt"] and r["first"] < 0)
                batch.append((q[r["gid"]], r["ctx"], 1, comp))
        total = self.cost(batch)
        xfer = float(moved * b * KV_TOKEN) * self.inv_link
        if xfer > 0:
            total = max(total, xfer) if self.overlap else total + xfer
        t_end = t + max(1, math.ceil(total))
        self.iters += 1
        self.peak = max(self.peak, used)
        self.ubns = self.ubns + used * (t_end - t)
        out = []
        for r in run:
            if r["gid"] in idle:
                continue
            if r["ctx"] >= r["tgt"]:
                r["ctx"] += 1
                r["gd"] += 1
                r["gap"] = max(r["gap"], t_end - r["last"])
                r["last"] = t_end
                self.dec_tok += 1
                if r["gd"] == r["o"]:
                    r.update(ph="done", fin=t_end)
            elif q.get(r["gid"], 0) > 0:
                r["ctx"] += q[r["gid"]]
                self.pre_tok += q[r["gid"]]
                if r["ctx"] == r["tgt"] and r["first"] < 0:
                    r["first"] = r["last"] = t_end
                    if self.prefill:
                        r["ph"] = "out"
                        out.append(r)
        self.clock = t_end
        return out


def _req(gid, at, p, o, **kw):
    r = dict(gid=gid, at=at, p=p, o=o, ph="new", ctx=0, tgt=p, gd=0, seq=None, admit=-1,
             first=-1, last=-1, gap=0, npre=0, fin=-1, sw=False, fresh=True)
    r.update(kw)
    return r


def brute_pd(reqs, n_p, n_d, NBp, NBd, b, M, K, cost_p, cost_d, link_bw, permille=0,
             swap_bw=0.0, overlap=0):
    """Global event loop over n_p prefill and n_d decode devices."""
    P = [Device(True, NBp, b, M, K, cost_p) for _ in range(n_p)]
    D = [Device(False, NBd, b, M, K, cost_d, permille, swap_bw, overlap) for _ in range(n_d)]
    cap_d = NBd * permille // 1000 if permille else NBd
    rej = set()
    for i, (a, p, o) in enumerate(reqs):
        if NBp == 0 or NBd == 0 or blocks(p, b) > NBp or blocks(p + o, b) > NBd or \
                blocks(p + 1, b) > cap_d:
            rej.add(i)
        else:
            P[i % n_p].reqs.append(_req(i, a, p, o))
    link_free = [0] * n_p
    devs = P + D
    while True:
        starts = [(d.next_start(), k) for k, d in enumerate(devs) if d.next_start() is not None]
        if not starts:
            break
        s, k = min(starts)
        done = devs[k].iterate(s)
        for r in done:  # the prompt's KV crosses device k's link, in completion order
            x = 0 if link_bw == 0 else math.ceil(float(r["p"] * KV_TOKEN) * (1e9 / link_bw))
            link_free[k] = max(r["first"], link_free[k]) + x
            D[r["gid"] % n_d].reqs.append(_req(r["gid"], link_free[k], r["p"], r["o"],
                                               ctx=r["p"], first=r["first"], last=r["first"],
                                               admit=r["admit"]))
    recs = [(-1, -1, -1, 0, 0, 2) if i in rej else (-1, -1, -1, 0, 0, 0) for i in range(len(reqs))]
    for d in D:
        for r in d.reqs:
            if r["ph"] == "done":
                recs[r["gid"]] = (r["admit"], r["first"], r["fin"], r["gap"], r["npre"], 1)
    ub = 0.0
    for d in devs:
        ub = ub + d.ubns
    cnt = dict(n_iters=sum(d.iters for d in devs), n_preempt=sum(d.n_pre for d in D),
               prefill_tokens=sum(d.pre_tok for d in devs),
               decode_tokens=sum(d.dec_tok for d in D),
               peak_used_blocks=max(d.peak for d in D), used_block_ns=ub)
    return recs, cnt


def _trace(reqs):
    return {"arrival_ns": np.array([r[0] for r in reqs], np.int64),
            "prompt_len": np.array([r[1] for r in reqs], np.int32),
            "output_len": np.array([r[2] for r in reqs], np.int32)}


def _pd_point(F, BW, Fp, BWp, NBp, NBd, b, M, K, n_p, n_d, link_bw, permille=0, swap_bw=0.0,
              overlap=0):
    return dict(peak_flops=F, mem_bw=BW, capacity_bytes=max(1, NBd * b * KV_TOKEN),
                mem_util_permille=1000, block_size=b, max_batch=M, chunk_size=K,
                admit_mem_permille=permille, swap_bw=swap_bw, swap_overlap=overlap,
                n_prefill=n_p, n_decode=n_d, p_peak_flops=Fp, p_mem_bw=BWp,
                p_capacity_bytes=max(1, NBp * b * KV_TOKEN), kv_link_bw=link_bw)


@pytest.mark.parametrize("hw", ["unit", "roofline"])
def test_pd_oracle_matches_global_event_loop(oracle, hw):
    rnd = random.Random(77 if hw == "unit" else 78)
    F, BW = (1e300, 1e300) if hw == "unit" else (2e9, 1.5e9)
    Fp, BWp = (1e300, 1e300) if hw == "unit" else (3e9, 1e9)
    cost_d = lambda batch: oracle.iter_total(TOY, 1e9 / F, 1e9 / BW, batch)
    cost_p = lambda batch: oracle.iter_total(TOY, 1e9 / Fp, 1e9 / BWp, batch)
    seen_pre = seen_swap = seen_wait = 0
    for case in range(400 if hw == "unit" else 150):
        n = rnd.randint(1, 14)
        b = rnd.choice([1, 2, 3, 4])
        M = rnd.choice([1, 2, 3, 5])
        K = rnd.choice([0, 0, M, M + 2])
        NBd, NBp = rnd.randint(1, 14), rnd.randint(1, 10)
        n_p, n_d = rnd.randint(1, 3), rnd.randint(1, 3)
        permille = rnd.choice([0, 0, 500, 1000])
        swap_bw = rnd.choice([0.0, 0.0, 2e8, 2e9])
        overlap = rnd.choice([0, 1])
        link_bw = rnd.choice([0.0, 16e9, 1.6e9, 4e8])
        t, reqs = 0, []
        for _ in range(n):
            t += rnd.choice([0, 0, 1, 2, 5, 40])
            reqs.append((t, rnd.randint(1, 9), rnd.randint(1, 6)))
        pt = _pd_point(F, BW, Fp, BWp, NBp, NBd, b, M, K, n_p, n_d, link_bw, permille, swap_bw,
                       overlap)
        out, req, _, viol = oracle.simulate_point(TOY, _trace(reqs), pt)
        assert viol == 0, case
        want, cnt = brute_pd(reqs, n_p, n_d, NBp, NBd, b, M, K, cost_p, cost_d, link_bw,
                             permille, swap_bw, overlap)
        got = [tuple(int(x) for x in r) for r in req]
        assert got == want, (case, reqs, pt)
        for k, v in cnt.items():
            assert out[k] == v, (k, case, pt)
        assert out["n_done"] == sum(1 for r in want if r[5] == 1)
        assert out["n_rejected"] == sum(1 for r in want if r[5] == 2)
        seen_pre += cnt["n_preempt"]
        seen_swap += cnt["n_preempt"] if swap_bw > 0 else 0
        # a request that waited on its decode device: gap above one iteration
        seen_wait += sum(1 for r in want if r[5] == 1 and r[3] > 1)
    assert seen_pre > 10 and seen_swap > 3 and seen_wait > 20


A100 = dict(peak_flops=312e12, mem_bw=2.0e12, capacity_bytes=80_000_000_000,
            mem_util_permille=900, block_size=16, max_batch=32, chunk_size=0)


def test_pd_single_request_closed_form(oracle):
    """One request alone: TTFT is its prefill on the prefill device, its KV
    takes ceil(bytes / link bandwidth), then each decode is one batch-of-one
    iteration on the decode device; the first decode's gap spans the
    transfer."""
    from paper_2503_08415_amd import workloads as W
    m = W.MODELS["llama2-7b"]
    pt = dict(A100, n_prefill=1, n_decode=1, p_peak_flops=989e12, p_mem_bw=3.35e12,
              p_capacity_bytes=80_000_000_000, kv_link_bw=25e9)
    dd = oracle.derive(m, pt)
    dp = oracle.derive(m, dict(pt, peak_flops=989e12, mem_bw=3.35e12))
    for arr, p, o in [(0, 1, 1), (5_000, 700, 9), (123_456_789, 3000, 40)]:
        out, req, _, viol = oracle.simulate_point(m, _trace([(arr, p, o)]), pt)
        assert viol == 0
        first = arr + oracle.iter_ns(m, dp["inv_flops_ns"], dp["inv_bw_ns"], [(p, 0, 1, 1)])
        kv = math.ceil(float(p * dd["kv_bytes_per_token"]) * (1e9 / 25e9))
        t, gap = first + kv, 0
        for k in range(o):
            c = oracle.iter_ns(m, dd["inv_flops_ns"], dd["inv_bw_ns"], [(1, p + k, 0, 0)])
            gap = max(gap, t + c - (first if k == 0 else t))
            t += c
        r = req[0]
        assert (int(r["admit_ns"]), int(r["first_token_ns"]), int(r["finish_ns"]),
                int(r["max_gap_ns"]), int(r["status"])) == (arr, first, t, gap, 1)
        assert out["n_iters"] == 1 + o and out["decode_tokens"] == o
        assert out["prefill_tokens"] == p


def test_pd_ttft_depends_only_on_prefill_devices(oracle):
    """Round robin over two prefill devices: every request's admission and
    first token equal those of a one-prefill-device point run over its own
    device's share of the trace, whatever the decode side does."""
    from paper_2503_08415_amd import workloads as W
    m = W.MODELS["llama2-7b"]
    tr = W.make_trace({"arrival": ("poisson", 12.0), "prompt": ("uniform", 16, 2048),
                       "output": ("uniform", 4, 300)}, 300, 4242)
    pt = dict(A100, capacity_bytes=24_000_000_000, chunk_size=512, n_prefill=2, n_decode=3,
              p_peak_flops=200e12, p_mem_bw=1.5e12, p_capacity_bytes=20_000_000_000,
              kv_link_bw=10e9)
    _, req, _, _ = oracle.simulate_point(m, tr, pt)
    for w in range(2):
        sub = {k: v[w::2] for k, v in tr.items()}
        _, req1, _, _ = oracle.simulate_point(m, sub, dict(pt, n_prefill=1))
        assert np.array_equal(req["first_token_ns"][w::2], req1["first_token_ns"])
        assert np.array_equal(req["admit_ns"][w::2], req1["admit_ns"])


def test_pd_more_decode_devices_never_delay_first_tokens_and_relieve_memory(oracle):
    """Adding decode devices changes nothing before the KV transfer, and
    under memory pressure it lowers the preemption count."""
    from paper_2503_08415_amd import workloads as W
    m = W.MODELS["llama2-7b"]
    tr = W.make_trace({"arrival": ("poisson", 6.0), "prompt": ("lognormal", 5.5, 1.0, 4, 4096),
                       "output": ("lognormal", 5.0, 0.9, 1, 2048)}, 400, 99)
    pt = dict(A100, capacity_bytes=20_000_000_000, n_prefill=1, n_decode=1,
              p_peak_flops=312e12, p_mem_bw=2e12, p_capacity_bytes=80_000_000_000,
              kv_link_bw=25e9)
    out1, req1, _, _ = oracle.simulate_point(m, tr, pt)
    out3, req3, _, _ = oracle.simulate_point(m, tr, dict(pt, n_decode=3))
    assert np.array_equal(req1["first_token_ns"], req3["first_token_ns"])
    assert out1["n_preempt"] > 0 and out3["n_preempt"] < out1["n_preempt"]
    assert out3["sum_e2e_ns"] < out1["sum_e2e_ns"]


def test_pd_bad_arguments(oracle):
    tr = _trace([(0, 4, 2)])
    base = _pd_point(1e12, 1e12, 1e12, 1e12, 8, 8, 2, 4, 0, 1, 1, 1e9)
    for bad in (dict(n_prefill=0), dict(n_decode=0), dict(n_prefill=17), dict(n_decode=17),
                dict(policy=1), dict(policy=2), dict(p_peak_flops=0.0),
                dict(p_mem_bw=float("nan")), dict(p_capacity_bytes=0),
                dict(kv_link_bw=-1.0), dict(kv_link_bw=float("inf"))):
        with pytest.raises(oracle.OracleError):
            oracle.simulate_point(TOY, tr, dict(base, **bad))
