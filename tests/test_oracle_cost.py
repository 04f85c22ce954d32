"""Pins for the oracle's block budget and per-operator roofline cost model.

The paper gives no cost formula (its compute simulator is described as
operator-level and transformer-oriented, Sec. III overview; prefill is
compute-bound and decode memory-bound, Sec. II-A).  The oracle's reading is
pinned here against values fixed outside the oracle: published model sizes,
hand-computed toy-model costs, textbook limits, and exact rational
arithmetic for the fp64 rounding.
"""
import json
import math
import os
import random
from fractions import Fraction

import pytest

from paper_2503_08415_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _pt(**kw):
    base = dict(peak_flops=1e12, mem_bw=1e12, capacity_bytes=10**12, mem_util_permille=1000,
                block_size=16, max_batch=1, chunk_size=0)
    base.update(kw)
    return base


def test_weight_and_kv_bytes_match_published_sizes(oracle):
    g = _load("model_sizes.json")["models"]
    for name, ref in g.items():
        m = W.MODELS[name]
        d = oracle.derive(m, _pt())
        norms = (2 * m["n_layers"] + 1) * m["d_model"]
        assert d["weight_bytes"] == 2 * (ref["params"] - norms), name
        assert d["kv_bytes_per_token"] == ref["kv_bytes_per_token"], name


def test_block_budget_from_published_sizes(oracle):
    sizes = _load("model_sizes.json")["models"]

    def nb(model, cap, util, b):
        m = W.MODELS[model]
        w = 2 * (sizes[model]["params"] - (2 * m["n_layers"] + 1) * m["d_model"])
        budget = cap * util // 1000 - (w if m["weights_in_capacity"] else 0)
        return max(0, budget // (b * sizes[model]["kv_bytes_per_token"]))

    cases = [("llama2-7b", 80_000_000_000, 900, 16),
             ("llama2-13b", 40_000_000_000, 900, 16),
             ("llama2-13b", 288_000_000_000, 900, 8),
             ("llama2-70b-kvonly", 24_000_000_000, 1000, 16),
             ("gqa-7b", 288_000_000_000, 900, 8),
             ("llama2-13b", 20_000_000_000, 900, 16)]  # weights exceed capacity -> 0
    for model, cap, util, b in cases:
        d = oracle.derive(W.MODELS[model], _pt(capacity_bytes=cap, mem_util_permille=util,
                                                block_size=b))
        assert d["num_blocks"] == nb(model, cap, util, b), (model, cap, b)
    # the 7B / 80 GB / 16-token-block configuration holds 6976 blocks
    assert oracle.derive(W.MODELS["llama2-7b"], _pt(capacity_bytes=80_000_000_000,
                                                    mem_util_permille=900))["num_blocks"] == 6976


def test_toy_model_hand_values(oracle):
    g = _load("cost_toy.json")
    m = g["model"]
    for case in g["cases"]:
        iF, iB = 1e9 / case["peak_flops"], 1e9 / case["mem_bw"]
        assert oracle.iter_ns(m, iF, iB, g["batch"]) == case["iter_ns"], case["note"]
        # the per-operator values add up as the fixture says
        ops = case["op_ns"]
        if case["iter_ns"] > 1:
            assert sum(ops[:6]) * m["n_layers"] + ops[6] == case["iter_ns"]
    for case in g["extra_batches"]:
        iF, iB = 1e9 / case["peak_flops"], 1e9 / case["mem_bw"]
        assert oracle.iter_ns(m, iF, iB, case["batch"]) == case["iter_ns"], case["name"]


def _exact_iter(m, F, BW, batch):
    """Exact rational iteration time of the roofline reading (rounding pin)."""
    L, d, h, hkv = m["n_layers"], m["d_model"], m["n_heads"], m["n_kv_heads"]
    dkv = hkv * (d // h)
    f, g, V, e, ekv = m["ffn_dim"], 1 + m["ffn_gated"], m["vocab"], m["w_bytes"], m["kv_bytes"]
    T = TP = AP = CP = nD = CD = R = 0
    for q, c0, pf, comp in batch:
        if pf:
            T += q; TP += q; AP += q * c0 + q * (q + 1) // 2; CP += c0 + q; R += comp
        else:
            T += 1; nD += 1; CD += c0 + 1; R += 1
    iF, iB = Fraction(10**9) / Fraction(F), Fraction(10**9) / Fraction(BW)
    ops = [(2*T*d*(d+2*dkv), e*(d*(d+2*dkv)+T*d)+ekv*T*2*dkv+e*T*d),
           (4*d*AP, ekv*2*dkv*CP+e*2*d*TP), (4*d*CD, ekv*2*dkv*CD+e*2*d*nD),
           (2*T*d*d, e*(d*d+2*T*d)), (2*g*T*d*f, e*(g*d*f+T*d+g*T*f)), (2*T*f*d, e*(f*d+T*f+T*d))]
    layer = sum(max(a * iF, b * iB) for a, b in ops)
    lm = max(2*R*d*V*iF, e*(d*V+R*d+R*V)*iB) if R else 0
    return L * layer + lm


def test_fp64_rounding_matches_exact_arithmetic(oracle):
    rnd = random.Random(7)
    m = W.MODELS["llama2-7b"]
    for _ in range(300):
        F = rnd.choice(W.FLOPS_GRID8) * rnd.uniform(0.5, 2)
        BW = rnd.choice(W.BW_GRID8) * rnd.uniform(0.5, 2)
        batch = []
        for _ in range(rnd.randint(1, 6)):
            if rnd.random() < 0.5:
                batch.append((1, rnd.randint(0, 4000), 0, 0))
            else:
                batch.append((rnd.randint(1, 2048), rnd.randint(0, 4000), 1, rnd.randint(0, 1)))
        exact = _exact_iter(m, F, BW, batch)
        got = oracle.iter_ns(m, 1e9 / F, 1e9 / BW, batch)
        want = max(1, math.ceil(exact))
        frac = exact - math.floor(exact)
        if 1e-6 < frac < 1 - 1e-6:
            assert got == want
        else:
            assert abs(got - want) <= 1


def test_decode_limit_is_weight_bytes_over_bandwidth(oracle):
    """Decode at batch 1 with unbounded compute: the iteration streams every
    matmul weight plus the LM head once (Sec. II-A: decode is memory-bound)."""
    sizes = _load("model_sizes.json")["models"]
    for name in ("llama2-7b", "gqa-7b", "llama2-70b-kvonly"):
        m = W.MODELS[name]
        L, d, V = m["n_layers"], m["d_model"], m["vocab"]
        streamed = 2 * (sizes[name]["params"] - (2 * L + 1) * d - V * d)  # no embedding table
        BW = 2e12
        t = oracle.iter_ns(m, 1e9 / 1e300, 1e9 / BW, [(1, 0, 0, 0)])
        floor_ns = streamed * 1e9 / BW
        # activations of one token are < 64 KiB per operator
        assert floor_ns <= t <= floor_ns + (L * 6 + 1) * 65536 * 1e9 / BW + 1


def test_decode_slope_is_kv_bytes_per_token(oracle):
    """Each extra context token read by a decode costs its KV bytes."""
    sizes = _load("model_sizes.json")["models"]
    for name in ("llama2-7b", "gqa-7b", "llama2-13b"):
        m = W.MODELS[name]
        BW = 2e12
        t0 = oracle.iter_ns(m, 0.0, 1e9 / BW, [(1, 100, 0, 0)])
        t1 = oracle.iter_ns(m, 0.0, 1e9 / BW, [(1, 1100, 0, 0)])
        want = sizes[name]["kv_bytes_per_token"] * 1000 * 1e9 / BW
        assert abs((t1 - t0) - want) <= 2


def test_prefill_limit_is_two_flops_per_parameter_per_token(oracle):
    """Prefill with unbounded bandwidth: 2 FLOPs per matmul parameter per
    token, plus causal attention and one LM-head row (Sec. II-A: prefill is
    compute-bound)."""
    sizes = _load("model_sizes.json")["models"]
    for name in ("llama2-7b", "llama2-13b"):
        m = W.MODELS[name]
        L, d, V = m["n_layers"], m["d_model"], m["vocab"]
        n_matmul = sizes[name]["params"] - (2 * L + 1) * d - 2 * V * d
        F = 312e12
        for p in (1, 128, 1024, 4096):
            flops = 2 * n_matmul * p + 4 * d * L * (p * (p + 1) // 2) + 2 * d * V
            t = oracle.iter_ns(m, 1e9 / F, 0.0, [(p, 0, 1, 1)])
            assert abs(t - flops * 1e9 / F) <= 2, (name, p)


def test_gqa_changes_only_attention_and_qkv(oracle):
    """With the same d, grouped KV heads shrink K/V projections and KV reads
    only: FFN-dominated prefill time moves by exactly the QKV FLOP change."""
    mha = dict(W.MODELS["llama2-7b"], ffn_dim=14336)
    gqa = dict(mha, n_kv_heads=8)
    F = 1e15
    for p in (64, 512):
        tm = oracle.iter_ns(mha, 1e9 / F, 0.0, [(p, 0, 1, 0)])
        tg = oracle.iter_ns(gqa, 1e9 / F, 0.0, [(p, 0, 1, 0)])
        d, L = 4096, 32
        dq = 2 * p * d * (2 * d - 2 * 1024) * L  # QKV FLOPs removed by GQA
        assert abs((tm - tg) - dq * 1e9 / F) <= 2


def test_infinitely_fast_hardware_floor(oracle):
    m = W.MODELS["gqa-7b"]
    assert oracle.iter_ns(m, 1e9 / 1e300, 1e9 / 1e300, [(2048, 30000, 1, 1)] * 4) == 1


def test_realistic_scale_iteration_times(oracle):
    """LLaMA2-7B on 312 TFLOP/s and 2 TB/s: a batch-1 decode, a batch-64
    decode and a 1024-token prefill, against values computed outside this
    repository's code (tests/golden/cost_7b_scale.json, Sec. II-A)."""
    g = _load("cost_7b_scale.json")
    m = W.MODELS["llama2-7b"]
    iF = 1e9 / g["hardware"]["peak_flops"]
    iB = 1e9 / g["hardware"]["mem_bw"]
    for c in g["cases"]:
        if "batch_repeat" in c:
            row, k = c["batch_repeat"]
            batch = [tuple(row)] * k
        else:
            batch = [tuple(r) for r in c["batch"]]
        assert oracle.iter_ns(m, iF, iB, batch) == c["iter_ns"], c["name"]
    # the batch-1 decode sits within 3 % of weights / bandwidth (Sec. II-A)
    w = oracle.derive(m, _pt())["weight_bytes"]
    assert abs(g["cases"][0]["iter_ns"] - w * iB) < 0.03 * w * iB
