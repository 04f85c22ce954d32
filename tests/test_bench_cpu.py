"""Host-side checks of the benchmark contract and the synthetic workloads
(no GPU): the multi-GPU refusal, the seeded generators' determinism, and the
shapes each named sweep promises."""
import os
import subprocess
import sys

import numpy as np
import pytest

from paper_2503_08415_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.mark.parametrize("name", ["c1", "c2", "c6", "c7", "c8", "u1"])
def test_workloads_are_seeded_and_shaped(name):
    m1, t1, p1 = W.make_config(name)
    m2, t2, p2 = W.make_config(name)
    assert m1 == m2 and len(t1) == len(t2)
    for a, b in zip(t1, t2):
        for k in ("arrival_ns", "prompt_len", "output_len"):
            assert np.array_equal(a[k], b[k])
        assert (np.diff(a["arrival_ns"]) >= 0).all()
        assert (a["prompt_len"] >= 1).all() and (a["output_len"] >= 1).all()
    for k in p1:
        assert np.array_equal(p1[k], p2[k])
    n = len(p1["peak_flops"])
    assert set(p1) == set(W.POINT_FIELDS)
    assert ((p1["trace_id"] >= 0) & (p1["trace_id"] < len(t1))).all()
    assert W.CONFIGS[name][2].startswith("%d " % n)  # the description names the point count


def test_c8_splits_an_eight_device_node():
    _, _, p = W.make_config("c8")
    assert ((p["n_prefill"] + p["n_decode"]) == 8).all()
    assert set(p["n_prefill"].tolist()) == {1, 2, 3, 4}
    assert (p["policy"] == 0).all() and (p["kv_link_bw"] > 0).all()


@pytest.mark.parametrize("base,wide,reps", [("c6", "c6x", 24), ("c7", "c7x", 26),
                                             ("c8", "c8x", 4)])
def test_gpu_filling_sweeps_replicate_the_studies(base, wide, reps):
    """The wide sweeps are their study's grid repeated over replicates with
    traces of their own: replicate 0 is the study itself, and every
    replicate's traces differ from the others'."""
    _, tb, pb = W.make_config(base)
    _, tw, pw = W.make_config(wide)
    nb, nt = len(pb["peak_flops"]), len(tb)
    assert len(pw["peak_flops"]) == reps * nb and len(tw) == reps * nt
    for k in pb:
        assert np.array_equal(pw[k][:nb], pb[k])
        if k != "trace_id":
            assert np.array_equal(pw[k].reshape(reps, nb), np.tile(pb[k], (reps, 1)))
    assert np.array_equal(pw["trace_id"].reshape(reps, nb),
                          pb["trace_id"][None, :] + nt * np.arange(reps)[:, None])
    for a, b in zip(tw[:nt], tb):
        assert np.array_equal(a["arrival_ns"], b["arrival_ns"])
    firsts = {int(t["arrival_ns"][0]) for t in tw}
    assert len(firsts) == len(tw)
    units = (pw["n_prefill"] + pw["n_decode"]).clip(min=1)
    assert int(units.sum()) >= 8192


def test_unique_trace_sweep_is_c4_with_one_trace_per_point():
    _, t4, p4 = W.make_config("c4")
    _, tu, pu = W.make_config("c4u")
    n = len(p4["peak_flops"])
    assert len(tu) == n and np.array_equal(pu["trace_id"], np.arange(n))
    for k in p4:
        if k != "trace_id":
            assert np.array_equal(pu[k], p4[k])
    assert all(len(t["arrival_ns"]) == 4000 for t in tu)
    # 16 bytes per record (arrival int64, prompt and output int32)
    assert sum(16 * len(t["arrival_ns"]) for t in tu) == 16384 * 4000 * 16
    # each point's trace is drawn at its row's rate: mean gap near 1 / rate
    for i in (0, n // 2, n - 1):
        rate = 4.0 * (p4["trace_id"][i] + 1)
        gap = tu[i]["arrival_ns"][-1] / 4000 / 1e9
        assert abs(gap * rate - 1.0) < 0.1


def test_u1_calibration_workload_is_one_steady_batch():
    _, t, p = W.make_config("u1")
    assert len(t) == 1 and len(p["peak_flops"]) == 8192
    tr = t[0]
    assert (tr["arrival_ns"] == 0).all() and len(tr["arrival_ns"]) == 64
    assert (tr["output_len"] == 4000).all() and (p["max_batch"] == 64).all()


def test_traffic_is_reported_only_for_the_profiled_sources(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    f = tmp_path / "traffic.md"
    f.write_text("```\nsources-sha256: %s\ntraffic-bytes: c5 sim_kernel<4,0> 2.5e+10\n```\n"
                 % bench.kernel_sources_sha256())
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.recorded_traffic("c5", "sim_kernel<4,0>") == 2.5e10
    assert bench.recorded_traffic("c5", "sim_kernel<1,0>") is None
    assert bench.recorded_traffic("c6", "sim_kernel<4,0>") is None
    # a change to a kernel source or the build flags voids the figure
    monkeypatch.setattr(bench, "kernel_sources_sha256", lambda: "0" * 64)
    assert bench.recorded_traffic("c5", "sim_kernel<4,0>") is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.md"))
    assert bench.recorded_traffic("c5", "sim_kernel<4,0>") is None


def test_build_flags_are_part_of_the_profiled_sources():
    sys.path.insert(0, ROOT)
    import bench
    assert "paper_2503_08415_amd/build.py" in bench.KERNEL_SOURCES
    assert all(os.path.exists(os.path.join(ROOT, p)) for p in bench.KERNEL_SOURCES)


def _manifest():
    import json
    with open(os.path.join(ROOT, "tests", "golden", "workload_sha256.json")) as f:
        return json.load(f)["configs"]


@pytest.mark.parametrize("name", sorted(W.CONFIGS))
def test_workload_bytes_match_committed_digests(name):
    """Every named workload generates exactly the committed bytes
    (tests/golden/make_workload_sha256.py wrote the digests)."""
    assert W.digests(*W.make_config(name)) == _manifest()[name]


def test_iteration_work_unit_is_frozen_to_the_u1_calibration():
    """U, the algorithmic VALU instructions per simulated iteration behind
    roofline.achieved, is 6.5 and never above what the committed u1 counter
    run measured per iteration of the cheapest path (it may only move down,
    with a new u1 profile)."""
    import re
    sys.path.insert(0, ROOT)
    import bench
    assert bench.U_ITER == 6.5
    with open(os.path.join(ROOT, "profiles", "sim_kernel_sq_counters_u1.md")) as f:
        text = f.read()
    m = re.search(r"\|\s*SQ_INSTS_VALU\s*\|\s*[0-9.e+]+\s*\|\s*([0-9.]+)\s*\|", text)
    assert m, "the u1 profile states SQ_INSTS_VALU per simulated iteration"
    assert bench.U_ITER <= float(m.group(1))
