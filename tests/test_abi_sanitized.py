"""The host-only ABI tests (tests/test_abi.py) against a build of the library
whose host code carries AddressSanitizer and UndefinedBehaviorSanitizer.

The sanitized library is built with hipcc (device code unchanged, sanitizer
flags scoped to the host pass) and loaded into a child Python process with
the clang ASan runtime preloaded; any sanitizer report aborts that process.
No kernel is launched: this runs on the CPU.
"""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build_module():
    spec = importlib.util.spec_from_file_location(
        "_optima_build", os.path.join(ROOT, "paper_2512_13886_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


PROBE = """
import ctypes, sys
import paper_2512_13886_amd as L
assert L.library_path() == sys.argv[1], L.library_path()
# the sanitizer runtime is live in this process
assert hasattr(ctypes.CDLL(None), "__asan_init")
print("sanitized library loaded:", L.library_path())
"""


@pytest.mark.slow
def test_abi_under_host_sanitizers():
    b = _build_module()
    if not os.path.exists(b.HIPCC):
        pytest.skip("hipcc is not installed")
    lib = b.build_sanitized(verbose=False)
    env = dict(os.environ)
    env.update({
        "OPTIMA_LIBRARY": lib,
        "LD_PRELOAD": b.asan_runtime(),
        # Python's own allocator pools hide heap errors from ASan; leaks of
        # the interpreter and the HIP runtime are not this library's.
        "PYTHONMALLOC": "malloc",
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "PYTHONPATH": ROOT,
    })
    r = subprocess.run([sys.executable, "-c", PROBE, lib], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join("tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out
