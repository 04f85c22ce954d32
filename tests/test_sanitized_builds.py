"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the host code
(CPU only): the oracle under its pins, and the HIP library's host-side
validation path, which rejects every invalid input before its first device
call.  Device code is never built with a sanitizer."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RUNNER = os.path.join(ROOT, "tests", "sanitize_runner.py")


def _run(which, lib, files, preload, timeout):
    env = dict(os.environ)
    env["LD_PRELOAD"] = ":".join(preload)
    # the interpreter's own allocations are not this code's leaks; any
    # error report aborts the run
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sys.executable, RUNNER, which, lib, *files], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=timeout)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert "passed" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr


def test_oracle_pins_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "libtso_asan.so")
    src = os.path.join(ROOT, "oracle", "tso.c")
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer",
                    "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    src, "-o", lib, "-lm", "-lpthread"], check=True)
    rt = [subprocess.run(["gcc", "-print-file-name=%s" % n], capture_output=True, text=True,
                         check=True).stdout.strip() for n in ("libasan.so", "libubsan.so")]
    files = ["tests/test_oracle_cost.py", "tests/test_oracle_sched.py",
             "tests/test_oracle_pd.py", "tests/test_oracle_bruteforce.py"]
    _run("oracle", lib, files, rt, timeout=600)


def test_host_validation_under_asan_ubsan(tmp_path):
    from paper_2503_08415_amd import build as B
    rt = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")
    if not rt:
        pytest.skip("no clang AddressSanitizer runtime")
    lib = str(tmp_path / "libts_sweep_asan.so")
    # host code only: each sanitizer flag applies to the host compilation
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-g",
                "-shared-libasan"]
    B.build(out=lib, extra_flags=host_san)
    _run("sweep", lib, ["tests/test_abi_cpu.py"], rt[:1], timeout=600)
