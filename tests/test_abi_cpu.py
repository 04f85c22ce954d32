"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every entry point the header declares, the binding's struct layouts match
the header, and invalid arguments are rejected before any device call."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2503_08415_amd import sweep as S
from paper_2503_08415_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ts_sweep.h")


@pytest.fixture(scope="module")
def L():
    from paper_2503_08415_amd import build as B
    if B.is_stale():
        B.build()
    return S.lib()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ts_\w+)\s*\(", src)))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert set(names) == set(S.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


def test_struct_layouts():
    assert C.sizeof(S.Model) == 40
    assert C.sizeof(S.Trace) == 32
    assert C.sizeof(S.Point) == 104
    assert C.sizeof(S.Options) == 48
    assert S.REQ_DTYPE.itemsize == 40
    assert S.POINT_DTYPE.itemsize == 176
    src = open(HEADER).read()
    assert "Per-point result: 176 bytes" in src and "40 bytes" in src
    assert "#define TS_ABI_VERSION 4" in src


def test_header_layout_matches_binding(tmp_path):
    """Every field offset and struct size the C compiler derives from the
    header equals the one the Python binding declares."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no host C compiler")
    structs = [("ts_model", S.Model), ("ts_trace", S.Trace), ("ts_point", S.Point),
               ("ts_options", S.Options), ("ts_point_result", S.POINT_DTYPE),
               ("ts_req_result", S.REQ_DTYPE)]
    want, lines = [], []
    for cname, py in structs:
        if isinstance(py, np.dtype):
            fields = [(n, py.fields[n][1]) for n in py.names]
            size = py.itemsize
        else:
            fields = [(f[0], getattr(py, f[0]).offset) for f in py._fields_]
            size = C.sizeof(py)
        want.append("%s %d" % (cname, size))
        lines.append('printf("%s %%zu\\n", sizeof(%s));' % (cname, cname))
        for n, off in fields:
            want.append("%s.%s %d" % (cname, n, off))
            lines.append('printf("%s.%s %%zu\\n", offsetof(%s, %s));' % (cname, n, cname, n))
    src = tmp_path / "layout.c"
    src.write_text("#include <stddef.h>\n#include <stdio.h>\n#include \"ts_sweep.h\"\n"
                   "int main(void) {\n" + "\n".join(lines) + "\nreturn 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    got = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    assert [g for g in got if g] == want


def test_status_strings(L):
    for rc in (0, -1, -2, -3, -4, -5, 7):
        assert isinstance(L.ts_status_str(rc), bytes)


def _create(L, model, traces, points, opt=None):
    h = C.c_void_p()
    tr = (S.Trace * max(1, len(traces)))()
    keep = []
    for k, t in enumerate(traces):
        a = np.ascontiguousarray(t["arrival_ns"], np.int64)
        p = np.ascontiguousarray(t["prompt_len"], np.int32)
        o = np.ascontiguousarray(t["output_len"], np.int32)
        keep += [a, p, o]
        tr[k] = S.Trace(a.ctypes.data, p.ctypes.data, o.ctypes.data, len(a))
    pts, n = S.points_array(points)
    rc = L.ts_sweep_create(C.byref(S.model_struct(model)), tr, len(traces), pts, n,
                           C.byref(opt) if opt is not None else None, C.byref(h))
    return rc, h


def _base():
    m, traces, pts = W.make_config("c1")
    return m, traces, pts


def _mod_points(pts, **kw):
    q = {k: v.copy() for k, v in pts.items()}
    for k, v in kw.items():
        if k in q:
            q[k][:] = v
        else:
            q[k] = np.full(len(q["peak_flops"]), v)
    return q


def test_invalid_arguments_fail_before_device(L):
    m, traces, pts = _base()
    bad_models = [dict(m, d_model=4095), dict(m, n_kv_heads=5), dict(m, n_layers=0),
                  dict(m, ffn_gated=2), dict(m, vocab=0)]
    for bm in bad_models:
        rc, h = _create(L, bm, traces, pts)
        assert rc == S.TS_ERR_ARG and not h.value
    for kw in (dict(block_size=0), dict(max_batch=0), dict(chunk_size=8),
               dict(trace_id=3), dict(mem_util_permille=0), dict(mem_util_permille=1001),
               dict(capacity_bytes=0), dict(peak_flops=float("nan")),
               dict(mem_bw=float("inf")), dict(peak_flops=-1.0),
               dict(policy=S.POLICY_PREFILL_FIRST, chunk_size=64),
               dict(admit_mem_permille=-1), dict(admit_mem_permille=1001),
               dict(swap_bw=-1.0), dict(swap_bw=float("inf")), dict(swap_overlap=2)):
        rc, h = _create(L, m, traces, _mod_points(pts, **kw))
        assert rc == S.TS_ERR_ARG, kw
    for kw in (dict(max_batch=257), dict(policy=3), dict(policy=-1)):
        rc, h = _create(L, m, traces, _mod_points(pts, **kw))
        assert rc == S.TS_ERR_UNSUPPORTED, kw
    # disaggregated points
    pd = dict(n_prefill=1, n_decode=1, p_peak_flops=1e12, p_mem_bw=1e12,
              p_capacity_bytes=80_000_000_000, kv_link_bw=1e9)
    for kw in (dict(n_decode=0), dict(n_prefill=0), dict(n_prefill=17), dict(n_decode=17),
               dict(n_prefill=-1), dict(policy=S.POLICY_STATIC), dict(p_peak_flops=0.0),
               dict(p_mem_bw=float("nan")), dict(p_capacity_bytes=0), dict(kv_link_bw=-1.0),
               dict(kv_link_bw=float("inf"))):
        rc, h = _create(L, m, traces, _mod_points(pts, **dict(pd, **kw)))
        assert rc == S.TS_ERR_ARG, kw
    unsorted = dict(traces[0])
    unsorted["arrival_ns"] = traces[0]["arrival_ns"][::-1].copy()
    rc, _ = _create(L, m, [unsorted], pts)
    assert rc == S.TS_ERR_ARG
    zero_len = dict(traces[0])
    zero_len["output_len"] = np.zeros_like(traces[0]["output_len"])
    rc, _ = _create(L, m, [zero_len], pts)
    assert rc == S.TS_ERR_ARG
    opt = S.Options(4, 0, 0, 0, 0, 0, 0, 0)  # unknown flag
    rc, _ = _create(L, m, traces, pts, opt)
    assert rc == S.TS_ERR_ARG
    opt = S.Options(S.F_PER_REQUEST | S.F_NO_TAKEOVER, 0, 0, 0, 0, 0, 0, 0)  # the known ones
    rc, h = _create(L, m, traces, pts, opt)
    assert rc in (S.TS_OK, S.TS_ERR_DEVICE)  # validation passed (no GPU here)
    if rc == S.TS_OK:
        L.ts_sweep_destroy(h)
    opt = S.Options(0, 0, 2, 0, 0, 0, 0, 0)  # sub-range beyond the points
    rc, _ = _create(L, m, traces, pts, opt)
    assert rc == S.TS_ERR_ARG
    rc = L.ts_sweep_create(None, None, 0, None, 0, None, None)
    assert rc == S.TS_ERR_ARG


def test_exact_range_guard(L):
    """A shape whose cost-model integers could pass 2^53 is refused."""
    m, traces, pts = _base()
    long = {"arrival_ns": np.zeros(1, np.int64), "prompt_len": np.full(1, 1 << 20, np.int32),
            "output_len": np.ones(1, np.int32)}
    big = dict(m, d_model=65536, n_heads=64, n_kv_heads=64, ffn_dim=262144)
    rc, _ = _create(L, big, [long], _mod_points(pts, max_batch=256, capacity_bytes=10**15))
    assert rc == S.TS_ERR_UNSUPPORTED
    # on the 7B shape with a chunked prefill budget the same trace stays exact
    rc, h = _create(L, m, [long], _mod_points(pts, capacity_bytes=10**15, max_batch=1,
                                              chunk_size=2048))
    assert rc in (S.TS_OK, S.TS_ERR_DEVICE)  # validation passed (no GPU here)
    if rc == S.TS_OK:
        L.ts_sweep_destroy(h)


def test_null_handle_calls(L):
    assert L.ts_sweep_run(None, None) == S.TS_ERR_ARG
    assert L.ts_sweep_results(None, None, None) == S.TS_ERR_ARG
    a, b = C.c_float(), C.c_float()
    assert L.ts_sweep_timing(None, C.byref(a), C.byref(b)) == S.TS_ERR_ARG
    L.ts_sweep_destroy(None)


def test_missing_library_fails_loudly():
    # the binding has no fallback: without the built library every call raises
    code = ("import sys; sys.path.insert(0, %r)\n"
            "from paper_2503_08415_amd import sweep as S\n"
            "S.LIB_PATH = '/nonexistent/libts_sweep.so'\n"
            "try:\n    S.lib()\nexcept RuntimeError as e:\n    print('raised', e)\n" % ROOT)
    import subprocess
    import sys
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.startswith("raised") and "not built" in r.stdout


def test_product_package_never_reaches_the_oracle():
    # the oracle is test infrastructure: no module of the package imports,
    # loads or names it as code
    pkg = os.path.join(ROOT, "paper_2503_08415_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if not f.endswith((".py", ".hip", ".h", ".c", ".cpp")):
                continue
            src = open(os.path.join(dirpath, f)).read()
            assert not re.search(r"^\s*(from|import)\s+oracle\b", src, flags=re.M), f
            assert "tso_" not in src and "libtso" not in src and "tso.h" not in src, f


def test_oracle_shares_no_code_with_the_hip_path():
    odir = os.path.join(ROOT, "oracle")
    for f in os.listdir(odir):
        if f.endswith((".py", ".c", ".h")):
            src = open(os.path.join(odir, f)).read()
            for name in ("paper_2503_08415_amd", "ts_sweep", "csrc", "sweep_internal"):
                assert name not in src, (f, name)


def test_static_entry_rejects_invalid_arguments_before_device(L):
    """ts_sweep_run_static validates like ts_sweep_create, before any device call."""
    m, traces, pts = _base()
    tr = (S.Trace * 1)()
    t = traces[0]
    a = np.ascontiguousarray(t["arrival_ns"], np.int64)
    p = np.ascontiguousarray(t["prompt_len"], np.int32)
    o = np.ascontiguousarray(t["output_len"], np.int32)
    tr[0] = S.Trace(a.ctypes.data, p.ctypes.data, o.ctypes.data, len(a))
    out = np.zeros(1, dtype=S.POINT_DTYPE)
    for bm, bp in ((dict(m, d_model=4095), pts), (m, _mod_points(pts, block_size=0)),
                   (m, _mod_points(pts, max_batch=0))):
        ps, n = S.points_array(bp)
        rc = L.ts_sweep_run_static(C.byref(S.model_struct(bm)), tr, 1, ps, n, None, None,
                                   C.c_void_p(out.ctypes.data), None)
        assert rc == S.TS_ERR_ARG
    ps, n = S.points_array(_mod_points(pts, max_batch=300))
    rc = L.ts_sweep_run_static(C.byref(S.model_struct(m)), tr, 1, ps, n, None, None,
                               C.c_void_p(out.ctypes.data), None)
    assert rc == S.TS_ERR_UNSUPPORTED
    assert L.ts_sweep_run_static(None, None, 0, None, 0, None, None, None, None) == S.TS_ERR_ARG
