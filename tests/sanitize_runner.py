"""Run test files against sanitizer builds (CPU only; started by
test_sanitized_builds.py in a child process with the sanitizer runtime
preloaded).

    python tests/sanitize_runner.py oracle <libtso.so> <test files...>
    python tests/sanitize_runner.py sweep <libts_sweep.so> <test files...>

Points the oracle's, or the HIP library's, ctypes loader at the given
shared object, checks that the process really mapped it, and runs pytest
on the given files."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main():
    which, path, files = sys.argv[1], os.path.abspath(sys.argv[2]), sys.argv[3:]
    if which == "oracle":
        from oracle import tso
        tso.build = lambda force=False: path
        tso.lib()
    else:
        from paper_2503_08415_amd import sweep
        sweep.LIB_PATH = path
        sweep.lib()
    with open("/proc/self/maps") as f:
        maps = f.read()
    if path not in maps:
        print("sanitizer build %s was not loaded" % path)
        return 3
    import pytest
    return pytest.main(["-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu", *files])


if __name__ == "__main__":
    sys.exit(main())
