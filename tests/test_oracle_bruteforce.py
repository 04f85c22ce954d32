"""Brute-force cross-check of the oracle's scheduler on tiny random inputs.

A second, deliberately different implementation of the same scheduling
reading: requests are dicts, the waiting set is re-sorted by
(arrival, index) every time it is read, the preemption victim is found as
the running request with the largest admission sequence number (not by list
position), and block needs are recomputed from token counts (never carried
incrementally).  Iteration costs come from the oracle's cost function, so
this checks how the loop composes batches, not the roofline arithmetic
(pinned separately).
"""
import math
import random

import numpy as np
import pytest

TOY = {"n_layers": 1, "d_model": 8, "n_heads": 2, "n_kv_heads": 1, "ffn_dim": 16,
       "ffn_gated": 1, "vocab": 10, "w_bytes": 2, "kv_bytes": 2, "weights_in_capacity": 0}
KV_DIM = TOY["n_kv_heads"] * TOY["d_model"] // TOY["n_heads"]  # K/V width per token


def blocks(tokens, b):
    return -(-tokens // b)


def brute(reqs, NB, b, M, K, cost, policy=0, permille=0, swap_bw=0.0, overlap=0):
    """reqs: list of (arrival, p, o), sorted by arrival.  Returns records and counters.

    policy 0: mixed continuous batching; 1: prefill-first (an iteration that
    can admit the waiting head only admits and prefills); 2: static batching
    (admit only into an empty running set).  permille > 0 keeps first
    admissions within floor(NB * permille / 1000) used blocks.
    swap_bw > 0: preemption swaps the victim's blocks to host memory (it
    keeps its tokens) and re-admission brings them back over a link of
    swap_bw bytes/s, the transfer added to the iteration (overlap 0) or
    overlapped with its compute (overlap 1).  cost(batch) is the unquantised
    compute time."""
    block_bytes = b * 2 * TOY["n_layers"] * KV_DIM * TOY["kv_bytes"]
    inv_link = 1e9 / swap_bw if swap_bw > 0 else 0.0
    N = len(reqs)
    cap = NB * permille // 1000 if permille else NB
    reserve = NB - cap
    st = []
    for i, (a, p, o) in enumerate(reqs):
        rej = NB == 0 or blocks(p + o, b) > NB or blocks(p, b) > cap
        st.append(dict(i=i, a=a, p=p, o=o, ph="rej" if rej else "future", ctx=0, tgt=p,
                       gd=0, seq=None, admit=-1, first=-1, last=-1, gap=0, npre=0, fin=-1,
                       sw=False))
    t, nxt, seq, iters = 0, 0, 0, 0
    pre_tok = dec_tok = n_pre = 0

    def held(r):
        return blocks(max(r["ctx"], r["tgt"]), b)

    def running():
        return sorted([r for r in st if r["ph"] == "run"], key=lambda r: r["seq"])

    def waiting():
        return sorted([r for r in st if r["ph"] == "wait"], key=lambda r: (r["a"], r["i"]))

    def free():
        return NB - sum(held(r) for r in st if r["ph"] == "run")

    while NB > 0:
        while nxt < N and st[nxt]["a"] <= t:
            if st[nxt]["ph"] != "rej":
                st[nxt]["ph"] = "wait"
            nxt += 1
        if not running() and not waiting():
            if nxt == N:
                break
            t = st[nxt]["a"]
            continue
        preempted = False
        grow = set()  # requests holding one extra (reserved) block this iteration

        def room_for(h):
            return free() - len(grow) - (reserve if h["admit"] < 0 else 0)

        def need_of(h):  # a swapped request brings back every block it held
            return held(h) if h["sw"] else blocks(h["tgt"], b)

        moved = 0  # blocks swapped out or in this iteration
        pf = False
        if policy == 1 and waiting() and len(running()) < M:
            pf = need_of(waiting()[0]) <= room_for(waiting()[0])
        for r in ([] if pf else running()):
            if r["ph"] != "run":
                continue
            if not (r["ctx"] >= r["tgt"] and r["ctx"] % b == 0):
                continue
            while free() - len(grow) == 0:
                v = max(running(), key=lambda x: x["seq"])
                if swap_bw > 0:
                    moved += held(v) + (1 if v["i"] in grow else 0)
                    v.update(ph="wait", sw=True, npre=v["npre"] + 1)
                else:
                    v.update(ph="wait", ctx=0, tgt=v["p"] + v["gd"], npre=v["npre"] + 1)
                grow.discard(v["i"])
                n_pre += 1
                preempted = True
                if v is r:
                    break
            if r["ph"] == "run":
                grow.add(r["i"])
        run = running()
        q = {}
        budget = None if K == 0 else K - sum(1 for r in run if r["ctx"] >= r["tgt"])
        for r in run:
            if r["ctx"] < r["tgt"]:
                need = r["tgt"] - r["ctx"]
                q[r["i"]] = need if budget is None else min(need, budget)
                if budget is not None:
                    budget -= q[r["i"]]
        paused = {r["i"] for r in run if pf and r["ctx"] >= r["tgt"]}
        may = not preempted
        if policy == 2 and run:
            may = False
        if policy == 1 and not pf:
            may = False
        swapped_in = set()
        if may:
            for h in waiting():
                if len(running()) >= M:
                    break
                if not h["sw"] and budget is not None and budget <= 0:
                    break
                if need_of(h) > room_for(h):
                    break
                seq += 1
                if h["sw"]:  # back from host memory; works from the next iteration
                    moved += need_of(h)
                    h.update(ph="run", seq=seq, sw=False)
                    swapped_in.add(h["i"])
                    continue
                h.update(ph="run", seq=seq)
                if h["admit"] < 0:
                    h["admit"] = t
                q[h["i"]] = h["tgt"] if budget is None else min(h["tgt"], budget)
                if budget is not None:
                    budget -= q[h["i"]]
        run = running()
        used = NB - free() + len(grow)
        batch = []
        paused |= swapped_in
        for r in run:
            if r["i"] in paused:
                continue
            if r["ctx"] >= r["tgt"]:
                batch.append((1, r["ctx"], 0, 0))
            elif q.get(r["i"], 0) > 0:
                comp = int(r["ctx"] + q[r["i"]] == r["tgt"] and r["first"] < 0)
                batch.append((q[r["i"]], r["ctx"], 1, comp))
        total = cost(batch)
        xfer = float(moved * block_bytes) * inv_link
        if xfer > 0:
            total = max(total, xfer) if overlap else total + xfer
        dt = max(1, math.ceil(total))
        t_end = t + dt
        iters += 1
        for r in run:
            if r["i"] in paused:
                continue
            if r["ctx"] >= r["tgt"]:
                r["ctx"] += 1
                r["gd"] += 1
                r["gap"] = max(r["gap"], t_end - r["last"])
                r["last"] = t_end
                dec_tok += 1
                if r["gd"] == r["o"]:
                    r.update(ph="done", fin=t_end)
            elif q.get(r["i"], 0) > 0:
                r["ctx"] += q[r["i"]]
                pre_tok += q[r["i"]]
                if r["ctx"] == r["tgt"] and r["first"] < 0:
                    r["first"] = r["last"] = t_end
        t = t_end
        assert used >= 0
    recs = []
    for r in st:
        if r["ph"] == "done":
            recs.append((r["admit"], r["first"], r["fin"], r["gap"], r["npre"], 1))
        elif r["ph"] == "rej":
            recs.append((-1, -1, -1, 0, 0, 2))
        else:
            recs.append((-1, -1, -1, 0, 0, 0))
    return recs, dict(n_iters=iters, n_preempt=n_pre, prefill_tokens=pre_tok,
                      decode_tokens=dec_tok)


def _random_case(rnd):
    n = rnd.randint(1, 12)
    b = rnd.choice([1, 2, 3, 4])
    M = rnd.choice([1, 2, 3, 5])
    K = rnd.choice([0, 0, M, M + 1, M + 4])
    NB = rnd.randint(1, 12)
    policy = rnd.choice([0, 0, 1, 2])
    if policy == 1:
        K = 0
    permille = rnd.choice([0, 0, 250, 500, 750, 1000])
    swap_bw = rnd.choice([0.0, 0.0, 2e7, 2e8, 2e9])
    overlap = rnd.choice([0, 1])
    t, reqs = 0, []
    for _ in range(n):
        t += rnd.choice([0, 0, 1, 2, 5, 40])
        reqs.append((t, rnd.randint(1, 9), rnd.randint(1, 6)))
    return reqs, NB, b, M, K, policy, permille, swap_bw, overlap


@pytest.mark.parametrize("hw", ["unit", "roofline"])
def test_oracle_matches_brute_force(oracle, hw):
    rnd = random.Random(1234 if hw == "unit" else 99)
    F, BW = (1e300, 1e300) if hw == "unit" else (2e9, 1.5e9)
    iF, iB = 1e9 / F, 1e9 / BW
    cost = lambda batch: oracle.iter_total(TOY, iF, iB, batch)
    n_pre_seen = n_swap_seen = 0
    seen = set()
    for case in range(600 if hw == "unit" else 200):
        reqs, NB, b, M, K, policy, permille, swap_bw, overlap = _random_case(rnd)
        seen.add((policy, permille > 0, swap_bw > 0))
        tr = {"arrival_ns": np.array([r[0] for r in reqs], np.int64),
              "prompt_len": np.array([r[1] for r in reqs], np.int32),
              "output_len": np.array([r[2] for r in reqs], np.int32)}
        pt = dict(peak_flops=F, mem_bw=BW, capacity_bytes=NB * b * 16, mem_util_permille=1000,
                  block_size=b, max_batch=M, chunk_size=K, policy=policy,
                  admit_mem_permille=permille, swap_bw=swap_bw, swap_overlap=overlap)
        out, req, _, viol = oracle.simulate_point(TOY, tr, pt)
        assert viol == 0
        want, cnt = brute(reqs, NB, b, M, K, cost, policy, permille, swap_bw, overlap)
        got = [tuple(int(x) for x in r) for r in req]
        assert got == want, (case, reqs, NB, b, M, K, policy, permille, swap_bw, overlap)
        for k, v in cnt.items():
            assert out[k] == v, (k, case)
        n_pre_seen += cnt["n_preempt"]
        n_swap_seen += cnt["n_preempt"] if swap_bw > 0 else 0
    assert n_pre_seen > 20 and n_swap_seen > 10  # the random cases do preempt, also by swap
    assert len(seen) == 12  # every policy, with and without the ratio and swapping
