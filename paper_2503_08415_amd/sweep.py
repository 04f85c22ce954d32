"""Python binding of the MI355X serving-simulation sweep (``include/ts_sweep.h``).

Argument marshalling only: every step of the simulation runs in the HIP
kernels of ``libts_sweep.so``.  There is no CPU fallback; if the library
has not been built, :func:`lib` raises.

PyTorch is used for streams: :meth:`Sweep.run` enqueues on
``torch.cuda.current_stream()`` unless a stream is given.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libts_sweep.so")

TS_OK, TS_ERR_ARG, TS_ERR_UNSUPPORTED, TS_ERR_OOM, TS_ERR_DEVICE, TS_ERR_STATE = 0, -1, -2, -3, -4, -5
POINT_OK, POINT_NO_KV, POINT_ITER_LIMIT, POINT_TIME_LIMIT = 0, 1, 2, 3
REQ_PENDING, REQ_DONE, REQ_REJECTED = 0, 1, 2
F_PER_REQUEST = 1
F_NO_TAKEOVER = 2
POLICY_MIXED, POLICY_PREFILL_FIRST, POLICY_STATIC = 0, 1, 2
MAX_BATCH = 256


class Model(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_layers", "d_model", "n_heads", "n_kv_heads", "ffn_dim", "ffn_gated", "vocab",
        "w_bytes", "kv_bytes", "weights_in_capacity")]


class Trace(C.Structure):
    _fields_ = [("arrival_ns", C.c_void_p), ("prompt_len", C.c_void_p),
                ("output_len", C.c_void_p), ("n", C.c_int32)]


class Point(C.Structure):
    _fields_ = [("peak_flops", C.c_double), ("mem_bw", C.c_double),
                ("capacity_bytes", C.c_int64), ("mem_util_permille", C.c_int32),
                ("block_size", C.c_int32), ("max_batch", C.c_int32),
                ("chunk_size", C.c_int32), ("trace_id", C.c_int32), ("policy", C.c_int32),
                ("admit_mem_permille", C.c_int32), ("swap_overlap", C.c_int32),
                ("swap_bw", C.c_double), ("n_prefill", C.c_int32), ("n_decode", C.c_int32),
                ("p_peak_flops", C.c_double), ("p_mem_bw", C.c_double),
                ("p_capacity_bytes", C.c_int64), ("kv_link_bw", C.c_double)]


# point fields a points dict may leave out, and their values then
POINT_DEFAULTS = {"policy": 0, "admit_mem_permille": 0, "swap_overlap": 0, "swap_bw": 0.0,
                  "n_prefill": 0, "n_decode": 0, "p_peak_flops": 0.0, "p_mem_bw": 0.0,
                  "p_capacity_bytes": 0, "kv_link_bw": 0.0}


class Options(C.Structure):
    _fields_ = [("flags", C.c_uint32), ("first_point", C.c_int32), ("n_points", C.c_int32),
                ("pad", C.c_int32), ("iter_cap", C.c_int64), ("slo_ttft_ns", C.c_int64),
                ("slo_tpot_ns", C.c_int64), ("point_time_limit_ms", C.c_int64)]


REQ_DTYPE = np.dtype([("admit_ns", "<i8"), ("first_token_ns", "<i8"), ("finish_ns", "<i8"),
                      ("max_gap_ns", "<i8"), ("n_preempt", "<i4"), ("status", "<i4")])

POINT_DTYPE = np.dtype([
    ("status", "<i4"), ("n_done", "<i4"), ("n_rejected", "<i4"), ("num_blocks", "<i4"),
    ("n_iters", "<i8"), ("n_preempt", "<i8"), ("prefill_tokens", "<i8"),
    ("decode_tokens", "<i8"), ("peak_used_blocks", "<i8"),
    ("first_arrival_ns", "<i8"), ("last_finish_ns", "<i8"), ("sum_ttft_ns", "<i8"),
    ("sum_e2e_ns", "<i8"), ("max_e2e_ns", "<i8"), ("sum_tpot_num_ns", "<i8"),
    ("p50_e2e_ns", "<i8"), ("p90_e2e_ns", "<i8"), ("p99_e2e_ns", "<i8"),
    ("p50_ttft_ns", "<i8"), ("p99_ttft_ns", "<i8"), ("slo_ok", "<i8"),
    ("used_block_ns", "<f8"), ("digest", "<u8"), ("slo_tpot_ok", "<i8")])

# every entry point declared in include/ts_sweep.h
EXPORTS = ("ts_sweep_create", "ts_sweep_run", "ts_sweep_results", "ts_sweep_shape",
           "ts_sweep_timing", "ts_sweep_kernel_timing", "ts_sweep_kernel_work",
           "ts_sweep_run_static",
           "ts_sweep_destroy", "ts_status_str")
STATIC_SCRATCH_BYTES = 64 << 20  # TS_STATIC_SCRATCH_BYTES
# simulation launches, 3 * stage + class: stages one-worker points, prefill
# devices, decode devices; classes max_batch <= 64, <= 128, <= 256
N_SIM_KERNELS = 9

_lib = None


class SweepError(RuntimeError):
    def __init__(self, rc: int, what: str):
        msg = lib().ts_status_str(rc).decode()
        super().__init__("%s failed: %s (%d)" % (what, msg, rc))
        self.rc = rc


def lib():
    """Load the built library (raises if it is missing: no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("HIP library %s is not built; run __graft_entry__.build()"
                               % LIB_PATH)
        L = C.CDLL(LIB_PATH)
        L.ts_sweep_create.argtypes = [C.POINTER(Model), C.POINTER(Trace), C.c_int32,
                                      C.POINTER(Point), C.c_int32, C.POINTER(Options),
                                      C.POINTER(C.c_void_p)]
        L.ts_sweep_create.restype = C.c_int
        L.ts_sweep_run.argtypes = [C.c_void_p, C.c_void_p]
        L.ts_sweep_run.restype = C.c_int
        L.ts_sweep_results.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        L.ts_sweep_results.restype = C.c_int
        L.ts_sweep_shape.argtypes = [C.c_void_p, C.POINTER(C.c_int32), C.POINTER(C.c_int32)]
        L.ts_sweep_shape.restype = C.c_int
        L.ts_sweep_timing.argtypes = [C.c_void_p, C.POINTER(C.c_float), C.POINTER(C.c_float)]
        L.ts_sweep_timing.restype = C.c_int
        L.ts_sweep_kernel_timing.argtypes = [C.c_void_p, C.POINTER(C.c_float),
                                             C.POINTER(C.c_int32)]
        L.ts_sweep_kernel_timing.restype = C.c_int
        L.ts_sweep_kernel_work.argtypes = [C.c_void_p, C.POINTER(C.c_int64)]
        L.ts_sweep_kernel_work.restype = C.c_int
        L.ts_sweep_run_static.argtypes = [C.POINTER(Model), C.POINTER(Trace), C.c_int32,
                                          C.POINTER(Point), C.c_int32, C.POINTER(Options),
                                          C.c_void_p, C.c_void_p, C.c_void_p]
        L.ts_sweep_run_static.restype = C.c_int
        L.ts_sweep_destroy.argtypes = [C.c_void_p]
        L.ts_sweep_destroy.restype = None
        L.ts_status_str.argtypes = [C.c_int]
        L.ts_status_str.restype = C.c_char_p
        _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != TS_OK:
        raise SweepError(rc, what)


def model_struct(m: dict) -> Model:
    return Model(*[int(m[f]) for f, _ in Model._fields_])


def points_array(points: dict):
    n = len(points["peak_flops"])
    arr = (Point * max(n, 1))()
    cols = []
    for name, ty in Point._fields_:
        conv = float if ty is C.c_double else int
        col = points.get(name)
        cols.append((conv, col, POINT_DEFAULTS.get(name)))
    for i in range(n):
        arr[i] = Point(*[conv(col[i]) if col is not None else conv(dflt)
                         for conv, col, dflt in cols])
    return arr, n


def _traces_array(traces):
    keep = []
    tr = (Trace * max(1, len(traces)))()
    for k, t in enumerate(traces):
        a = np.ascontiguousarray(t["arrival_ns"], dtype=np.int64)
        p = np.ascontiguousarray(t["prompt_len"], dtype=np.int32)
        o = np.ascontiguousarray(t["output_len"], dtype=np.int32)
        keep += [a, p, o]
        tr[k] = Trace(a.ctypes.data, p.ctypes.data, o.ctypes.data, len(a))
    return tr, keep


def run_static(model: dict, traces, points: dict, *, per_request: bool = False,
               first_point: int = 0, n_points: int = 0, iter_cap: int = 0,
               slo_ttft_ns: int = 0, slo_tpot_ns: int = 0, point_time_limit_ms: int = 0,
               takeover: bool = True, stream=None):
    """One whole sweep through ``ts_sweep_run_static`` (no device allocation;
    buffers in the library's static scratch).  Returns (points, requests or None)."""
    L = lib()
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream or 0)
    tr, keep = _traces_array(traces)
    pts, n = points_array(points)
    count = (n - int(first_point)) if int(n_points) == 0 else int(n_points)
    count = max(count, 0)
    max_n = max([len(t["arrival_ns"]) for t in traces] + [1])
    flags = (F_PER_REQUEST if per_request else 0) | (0 if takeover else F_NO_TAKEOVER)
    opt = Options(flags, int(first_point), int(n_points), 0,
                  int(iter_cap), int(slo_ttft_ns), int(slo_tpot_ns), int(point_time_limit_ms))
    out = np.zeros(max(count, 1), dtype=POINT_DTYPE)
    req = np.zeros((count, max_n), dtype=REQ_DTYPE) if per_request else None
    _check(L.ts_sweep_run_static(C.byref(model_struct(model)), tr, len(traces), pts, n,
                                 C.byref(opt), C.c_void_p(handle), out.ctypes.data,
                                 req.ctypes.data if req is not None else None),
           "ts_sweep_run_static")
    del keep
    return out[:count], req


class Sweep:
    """One uploaded sweep: ``create`` on construction, then ``run`` / ``results``."""

    def __init__(self, model: dict, traces, points: dict, *, per_request: bool = False,
                 first_point: int = 0, n_points: int = 0, iter_cap: int = 0,
                 slo_ttft_ns: int = 0, slo_tpot_ns: int = 0, point_time_limit_ms: int = 0,
                 takeover: bool = True):
        L = lib()
        self._h = C.c_void_p()
        tr, keep = _traces_array(traces)
        pts, n = points_array(points)
        flags = (F_PER_REQUEST if per_request else 0) | (0 if takeover else F_NO_TAKEOVER)
        opt = Options(flags, int(first_point), int(n_points), 0,
                      int(iter_cap), int(slo_ttft_ns), int(slo_tpot_ns),
                      int(point_time_limit_ms))
        _check(L.ts_sweep_create(C.byref(model_struct(model)), tr, len(traces), pts, n,
                                 C.byref(opt), C.byref(self._h)), "ts_sweep_create")
        np_, mn = C.c_int32(), C.c_int32()
        _check(L.ts_sweep_shape(self._h, C.byref(np_), C.byref(mn)), "ts_sweep_shape")
        self.n_points, self.max_n = np_.value, mn.value
        self.per_request = per_request

    def run(self, stream=None):
        """Enqueue the sweep on a HIP stream (default: torch's current stream)."""
        if stream is None:
            import torch
            stream = torch.cuda.current_stream()
        handle = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream or 0)
        _check(lib().ts_sweep_run(self._h, C.c_void_p(handle)), "ts_sweep_run")

    def results(self):
        """Wait for the last run; returns (points, requests or None)."""
        pts = np.zeros(max(self.n_points, 1), dtype=POINT_DTYPE)
        req = None
        if self.per_request:
            req = np.zeros((self.n_points, self.max_n), dtype=REQ_DTYPE)
        _check(lib().ts_sweep_results(self._h, pts.ctypes.data,
                                      req.ctypes.data if req is not None else None),
               "ts_sweep_results")
        return pts[:self.n_points], req

    def timing(self):
        """(simulation ms, statistics ms) of the last run, from HIP events."""
        a, b = C.c_float(), C.c_float()
        _check(lib().ts_sweep_timing(self._h, C.byref(a), C.byref(b)), "ts_sweep_timing")
        return a.value, b.value

    def kernel_timing(self):
        """Per simulation kernel: (ms, points) of the last run, from HIP events."""
        ms = (C.c_float * N_SIM_KERNELS)()
        n = (C.c_int32 * N_SIM_KERNELS)()
        _check(lib().ts_sweep_kernel_timing(self._h, ms, n), "ts_sweep_kernel_timing")
        return [(ms[k], n[k]) for k in range(N_SIM_KERNELS)]

    def kernel_work(self):
        """Per simulation kernel: simulated iterations of the points it completed."""
        it = (C.c_int64 * N_SIM_KERNELS)()
        _check(lib().ts_sweep_kernel_work(self._h, it), "ts_sweep_kernel_work")
        return [int(it[k]) for k in range(N_SIM_KERNELS)]

    def close(self):
        if self._h:
            lib().ts_sweep_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
