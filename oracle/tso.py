"""ctypes binding for the CPU oracle (``oracle/tso.c``).

TEST INFRASTRUCTURE ONLY: used by ``tests/``, the smoke check and the
benchmark's CPU-baseline leg.  The product path never imports this module.

Inputs are the plain arrays produced by the workload generators; outputs are
numpy structured arrays whose field names match the GPU library's result
records, so tests can compare them field by field.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tso.c")
_HDR = os.path.join(_HERE, "tso.h")
_LIB = os.path.join(_HERE, "libtso.so")

CFLAGS = ["-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-Wall", "-Wextra", "-Wno-unused-parameter"]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no contraction, no fast-math)."""
    stale = (not os.path.exists(_LIB) or
             os.path.getmtime(_LIB) < max(os.path.getmtime(_SRC), os.path.getmtime(_HDR)))
    if force or stale:
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm", "-lpthread"])
        os.replace(tmp, _LIB)
    return _LIB


class Model(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_layers", "d_model", "n_heads", "n_kv_heads", "ffn_dim", "ffn_gated", "vocab",
        "w_bytes", "kv_bytes", "weights_in_capacity")]


class Trace(C.Structure):
    _fields_ = [("arrival_ns", C.POINTER(C.c_int64)), ("prompt_len", C.POINTER(C.c_int32)),
                ("output_len", C.POINTER(C.c_int32)), ("n", C.c_int32)]


class Point(C.Structure):
    _fields_ = [("peak_flops", C.c_double), ("mem_bw", C.c_double),
                ("capacity_bytes", C.c_int64), ("mem_util_permille", C.c_int32),
                ("block_size", C.c_int32), ("max_batch", C.c_int32),
                ("chunk_size", C.c_int32), ("trace_id", C.c_int32), ("policy", C.c_int32),
                ("admit_mem_permille", C.c_int32), ("swap_overlap", C.c_int32),
                ("pad", C.c_int32), ("swap_bw", C.c_double),
                ("n_prefill", C.c_int32), ("n_decode", C.c_int32),
                ("p_peak_flops", C.c_double), ("p_mem_bw", C.c_double),
                ("p_capacity_bytes", C.c_int64), ("kv_link_bw", C.c_double)]

# optional point fields and their defaults (a missing key means the default)
_OPTIONAL = {"mem_util_permille": 1000, "chunk_size": 0, "trace_id": 0, "policy": 0,
             "admit_mem_permille": 0, "swap_overlap": 0, "pad": 0, "swap_bw": 0.0,
             "n_prefill": 0, "n_decode": 0, "p_peak_flops": 0.0, "p_mem_bw": 0.0,
             "p_capacity_bytes": 0, "kv_link_bw": 0.0}


def _make_point(get) -> "Point":
    vals = []
    for name, ty in Point._fields_:
        v = get(name)
        vals.append(float(v) if ty is C.c_double else int(v))
    return Point(*vals)


class Options(C.Structure):
    _fields_ = [("iter_cap", C.c_int64), ("slo_ttft_ns", C.c_int64),
                ("slo_tpot_ns", C.c_int64), ("n_threads", C.c_int32),
                ("check_invariants", C.c_int32)]


class Derived(C.Structure):
    _fields_ = [("kv_bytes_per_token", C.c_int64), ("weight_bytes", C.c_int64),
                ("kv_budget_bytes", C.c_int64), ("num_blocks", C.c_int32),
                ("pad", C.c_int32), ("inv_flops_ns", C.c_double), ("inv_bw_ns", C.c_double)]


REQ_DTYPE = np.dtype([("admit_ns", "<i8"), ("first_token_ns", "<i8"), ("finish_ns", "<i8"),
                      ("max_gap_ns", "<i8"), ("n_preempt", "<i4"), ("status", "<i4")])

POINT_OUT_DTYPE = np.dtype([
    ("status", "<i4"), ("n_done", "<i4"), ("n_rejected", "<i4"), ("num_blocks", "<i4"),
    ("n_iters", "<i8"), ("n_preempt", "<i8"), ("prefill_tokens", "<i8"),
    ("decode_tokens", "<i8"), ("peak_used_blocks", "<i8"),
    ("first_arrival_ns", "<i8"), ("last_finish_ns", "<i8"), ("sum_ttft_ns", "<i8"),
    ("sum_e2e_ns", "<i8"), ("max_e2e_ns", "<i8"), ("sum_tpot_num_ns", "<i8"),
    ("p50_e2e_ns", "<i8"), ("p90_e2e_ns", "<i8"), ("p99_e2e_ns", "<i8"),
    ("p50_ttft_ns", "<i8"), ("p99_ttft_ns", "<i8"), ("slo_ok", "<i8"),
    ("used_block_ns", "<f8"), ("digest", "<u8"), ("slo_tpot_ok", "<i8")])

ITER_DTYPE = np.dtype([("t_start", "<i8"), ("iter_ns", "<i8"), ("n_decode", "<i4"),
                       ("n_prefill", "<i4"), ("tokens", "<i4"), ("used_blocks", "<i4"),
                       ("n_running", "<i4"), ("n_preempted", "<i4"), ("n_admitted", "<i4"),
                       ("n_finished", "<i4")])

POINT_OK, POINT_NO_KV, POINT_ITER_LIMIT = 0, 1, 2
POLICY_MIXED, POLICY_PREFILL_FIRST, POLICY_STATIC = 0, 1, 2
REQ_PENDING, REQ_DONE, REQ_REJECTED = 0, 1, 2

_lib = None


def lib():
    global _lib
    if _lib is None:
        L = C.CDLL(build())
        L.tso_derive.argtypes = [C.POINTER(Model), C.POINTER(Point), C.POINTER(Derived)]
        L.tso_derive.restype = C.c_int
        L.tso_iter_ns.argtypes = [C.POINTER(Model), C.c_double, C.c_double, C.c_int32,
                                  C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.tso_iter_ns.restype = C.c_int64
        L.tso_iter_total.argtypes = L.tso_iter_ns.argtypes
        L.tso_iter_total.restype = C.c_double
        L.tso_simulate_point.argtypes = [
            C.POINTER(Model), C.POINTER(Trace), C.POINTER(Point), C.POINTER(Options),
            C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.POINTER(C.c_int64),
            C.POINTER(C.c_int64)]
        L.tso_simulate_point.restype = C.c_int
        L.tso_run_points.argtypes = [C.POINTER(Model), C.POINTER(Trace), C.c_int32,
                                     C.POINTER(Point), C.c_int32, C.POINTER(Options),
                                     C.c_void_p, C.c_void_p, C.c_int32]
        L.tso_run_points.restype = C.c_int
        L.tso_record_hash.argtypes = [C.c_int64, C.c_void_p]
        L.tso_record_hash.restype = C.c_uint64
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, rc):
        super().__init__("oracle returned %d" % rc)
        self.rc = rc


def _model(m: dict) -> Model:
    return Model(*[int(m[f]) for f, _ in Model._fields_])


def _point(pts: dict, i: int) -> Point:
    return _make_point(lambda f: pts[f][i] if f in pts else _OPTIONAL[f])


def _single_point(p: dict) -> Point:
    return _make_point(lambda f: p[f] if f in p else _OPTIONAL[f])


class _TraceKeep:
    """Holds contiguous copies of the trace arrays alive for a C call."""

    def __init__(self, traces):
        self.arrays = []
        self.structs = (Trace * max(1, len(traces)))()
        for k, tr in enumerate(traces):
            a = np.ascontiguousarray(tr["arrival_ns"], dtype=np.int64)
            p = np.ascontiguousarray(tr["prompt_len"], dtype=np.int32)
            o = np.ascontiguousarray(tr["output_len"], dtype=np.int32)
            self.arrays += [a, p, o]
            self.structs[k] = Trace(a.ctypes.data_as(C.POINTER(C.c_int64)),
                                    p.ctypes.data_as(C.POINTER(C.c_int32)),
                                    o.ctypes.data_as(C.POINTER(C.c_int32)), len(a))


def default_threads() -> int:
    """Threads across design points: the cores this process may run on, at
    most 16 (one GPU's share of a shared host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def _options(iter_cap=0, slo_ttft_ns=0, slo_tpot_ns=0, n_threads=0, check_invariants=0):
    if int(n_threads) <= 0:
        n_threads = default_threads()
    return Options(int(iter_cap), int(slo_ttft_ns), int(slo_tpot_ns), int(n_threads),
                   int(check_invariants))


def derive(model: dict, point: dict) -> dict:
    d = Derived()
    rc = lib().tso_derive(C.byref(_model(model)), C.byref(_single_point(point)), C.byref(d))
    if rc != 0:
        raise OracleError(rc)
    return {f: getattr(d, f) for f, _ in Derived._fields_ if f != "pad"}


def iter_ns(model: dict, inv_flops_ns: float, inv_bw_ns: float, batch) -> int:
    """Cost of one iteration; ``batch`` = list of (q, c0, is_prefill, completes)."""
    n = len(batch)
    cols = [np.ascontiguousarray([b[k] for b in batch] or [0], dtype=np.int32) for k in range(4)]
    return int(lib().tso_iter_ns(C.byref(_model(model)), float(inv_flops_ns), float(inv_bw_ns),
                                 n, *[c.ctypes.data for c in cols]))


def iter_total(model: dict, inv_flops_ns: float, inv_bw_ns: float, batch) -> float:
    """The same batch's compute time in ns before quantisation."""
    n = len(batch)
    cols = [np.ascontiguousarray([b[k] for b in batch] or [0], dtype=np.int32) for k in range(4)]
    return float(lib().tso_iter_total(C.byref(_model(model)), float(inv_flops_ns),
                                      float(inv_bw_ns), n, *[c.ctypes.data for c in cols]))


def simulate_point(model: dict, trace: dict, point: dict, *, iter_cap=0, slo_ttft_ns=0,
                   slo_tpot_ns=0, check_invariants=True, log_cap=0):
    """Simulate one design point.  Returns (point_out, requests, log, violations)."""
    keep = _TraceKeep([trace])
    n = len(keep.arrays[0])
    out = np.zeros(1, dtype=POINT_OUT_DTYPE)
    req = np.zeros(max(n, 1), dtype=REQ_DTYPE)
    log = np.zeros(max(int(log_cap), 1), dtype=ITER_DTYPE)
    nlog = C.c_int64(0)
    viol = C.c_int64(0)
    opt = _options(iter_cap, slo_ttft_ns, slo_tpot_ns, 1, int(bool(check_invariants)))
    rc = lib().tso_simulate_point(C.byref(_model(model)), C.byref(keep.structs[0]),
                                  C.byref(_single_point(point)), C.byref(opt),
                                  out.ctypes.data, req.ctypes.data, log.ctypes.data,
                                  int(log_cap), C.byref(nlog), C.byref(viol))
    if rc != 0:
        raise OracleError(rc)
    nl = min(int(nlog.value), int(log_cap))
    return out[0], req[:n], log[:nl], int(viol.value)


def run_points(model: dict, traces, points: dict, *, per_request=False, iter_cap=0,
               slo_ttft_ns=0, slo_tpot_ns=0, n_threads=0):
    """Simulate every design point (threads across points).

    Returns (point_out[n_points], requests[n_points, max_n] or None)."""
    keep = _TraceKeep(traces)
    n_points = len(points["peak_flops"])
    pts = (Point * max(1, n_points))()
    for i in range(n_points):
        pts[i] = _point(points, i)
    out = np.zeros(max(n_points, 1), dtype=POINT_OUT_DTYPE)
    max_n = max([len(t["arrival_ns"]) for t in traces] + [1])
    req = None
    if per_request:  # rows of shorter traces are padded with pending records
        req = np.zeros((n_points, max_n), dtype=REQ_DTYPE)
        req["admit_ns"] = req["first_token_ns"] = req["finish_ns"] = -1
    opt = _options(iter_cap, slo_ttft_ns, slo_tpot_ns, n_threads, 0)
    rc = lib().tso_run_points(C.byref(_model(model)), keep.structs, len(traces), pts, n_points,
                              C.byref(opt), out.ctypes.data,
                              req.ctypes.data if req is not None else None, max_n)
    if rc != 0:
        raise OracleError(rc)
    return out[:n_points], req


def record_hash(index: int, rec) -> int:
    r = np.zeros(1, dtype=REQ_DTYPE)
    r[0] = rec
    return int(lib().tso_record_hash(int(index), r.ctypes.data))
