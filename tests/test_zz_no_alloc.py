"""ts_sweep_run_static, the entry point that allocates no device memory
(every buffer in the library's static scratch), against the handle entry
points ts_sweep_create + ts_sweep_run + ts_sweep_results on the same inputs:
two calls in a row, the second with a smaller sweep, every point record and
every request record bit for bit, also for points handed between launches."""
import numpy as np
import pytest

from paper_2503_08415_amd import workloads as W

pytestmark = pytest.mark.gpu

CAP = 2_000_000  # iteration cap: the c2 points need a few hundred thousand at most


@pytest.fixture(scope="module")
def S():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2503_08415_amd import sweep
    sweep.lib()
    return sweep


def handle_run(S, m, traces, pts, per_request):
    sw = S.Sweep(m, traces, pts, per_request=per_request, iter_cap=CAP)
    try:
        sw.run()
        return sw.results()
    finally:
        sw.close()


def same(a, b, ra, rb):
    assert a.dtype == b.dtype and a.shape == b.shape
    assert a.tobytes() == b.tobytes()
    if ra is None:
        assert rb is None
    else:
        assert ra.shape == rb.shape and ra.tobytes() == rb.tobytes()


def test_static_entry_matches_handle_entry(S):
    import torch
    m, traces, pts = W.make_config("c2")
    print("call 1: c2, 256 points x 1000 requests, per request", flush=True)
    a, ra = S.run_static(m, traces, pts, per_request=True, iter_cap=CAP)
    b, rb = handle_run(S, m, traces, pts, True)
    same(a, b, ra, rb)
    assert (a["n_done"] == 1000).all()
    # a smaller sweep second, on another stream: 48 points of 400 requests
    m2, t2, p2 = W.make_config("c2", n_requests=400)
    p2 = W.subset_points(p2, np.arange(3, 256, 5)[:48])
    print("call 2: c2 subset, 48 points x 400 requests, per request", flush=True)
    c, rc_ = S.run_static(m2, t2, p2, per_request=True, iter_cap=CAP,
                          stream=torch.cuda.Stream())
    d, rd = handle_run(S, m2, t2, p2, True)
    same(c, d, rc_, rd)
    assert len(c) == 48 and rc_.shape == (48, 400)
    # without request records, on the default stream (NULL)
    m1, t1, p1 = W.make_config("c1")
    print("call 3: c1, point records only", flush=True)
    e, re_ = S.run_static(m1, t1, p1, iter_cap=CAP, stream=0)
    f, rf = handle_run(S, m1, t1, p1, False)
    same(e, f, re_, rf)
    # points wider than 64 slots under bursts: the 64-slot launch hands some
    # on to the wider ones with hand-over records (in the scratch too)
    rng = np.random.default_rng(3)
    burst = {"arrival_ns": np.zeros(300, np.int64),
             "prompt_len": rng.integers(16, 200, 300).astype(np.int32),
             "output_len": rng.integers(5, 60, 300).astype(np.int32)}
    spread = {"arrival_ns": np.sort(rng.integers(0, 3_000_000_000, 400)).astype(np.int64),
              "prompt_len": rng.integers(16, 2000, 400).astype(np.int32),
              "output_len": rng.integers(5, 300, 400).astype(np.int32)}
    rows = [(256, 0, 0), (100, 0, 0), (64, 0, 0), (256, 512, 0), (130, 256, 1), (256, 0, 1)]
    k = len(rows)
    p4 = {"peak_flops": np.full(k, 312e12), "mem_bw": np.full(k, 2e12),
          "capacity_bytes": np.full(k, 80_000_000_000, np.int64),
          "mem_util_permille": np.full(k, 900, np.int32), "block_size": np.full(k, 16, np.int32),
          "max_batch": np.array([r[0] for r in rows], np.int32),
          "chunk_size": np.array([r[1] for r in rows], np.int32),
          "trace_id": np.array([r[2] for r in rows], np.int32)}
    m4 = W.MODELS["llama2-7b"]
    print("call 4: 6 points wider than 64 slots, bursts of 300, per request", flush=True)
    g, rg = S.run_static(m4, [burst, spread], p4, per_request=True, iter_cap=CAP)
    h, rh = handle_run(S, m4, [burst, spread], p4, True)
    same(g, h, rg, rh)


def test_static_entry_limits(S):
    """A sweep beyond the static scratch is refused before any device work;
    request records without the flag are a call-order error."""
    import ctypes as C
    m, traces, pts = W.make_config("c3")  # latency arrays alone: 131 MB
    print("oversized: c3", flush=True)
    with pytest.raises(S.SweepError) as ei:
        S.run_static(m, traces, pts, iter_cap=CAP)
    assert ei.value.rc == S.TS_ERR_UNSUPPORTED
    assert "static scratch" in S.lib().ts_status_str(S.TS_ERR_UNSUPPORTED).decode()
    m1, t1, p1 = W.make_config("c1")
    tr, keep = S._traces_array(t1)
    pts1, n = S.points_array(p1)
    opt = S.Options(0, 0, 0, 0, CAP, 0, 0, 0)
    out = np.zeros(1, dtype=S.POINT_DTYPE)
    req = np.zeros((1, 64), dtype=S.REQ_DTYPE)
    rc = S.lib().ts_sweep_run_static(C.byref(S.model_struct(m1)), tr, 1, pts1, n, C.byref(opt),
                                     None, C.c_void_p(out.ctypes.data),
                                     C.c_void_p(req.ctypes.data))
    assert rc == S.TS_ERR_STATE
    # the scratch is still usable after the refusals
    e, _ = S.run_static(m1, t1, p1, iter_cap=CAP)
    assert e["n_done"][0] == 64
