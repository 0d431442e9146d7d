"""The C ABI's host-side validation code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only).  A second copy of the library is built with the host pass instrumented
(paper_2606_01563_amd/build.py, sanitize=True; device code as usual) and tests/test_abi.py
runs against it in a child process with the sanitizer runtime preloaded.  Every call there
fails validation or is a size query, so nothing is launched; any out-of-bounds access,
use-after-free, signed overflow or other undefined behaviour on those paths aborts the child.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def _stale(lib, csrc):
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    srcs = glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.cpp")) + \
        glob.glob(os.path.join(csrc, "*.h")) + glob.glob(os.path.join(ROOT, "include", "*.h"))
    return any(os.path.getmtime(s) > t for s in srcs)


def test_abi_checks_pass_under_host_asan_and_ubsan():
    from paper_2606_01563_amd import build as B
    rt = _asan_runtime()
    if rt is None or not os.path.exists(B.HIPCC):
        pytest.skip("no hipcc or clang sanitizer runtime in this environment")
    lib = B.LIB_SAN
    if _stale(lib, B.CSRC):
        B.build(sanitize=True)
    env = dict(os.environ, LD_PRELOAD=rt, MKV_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi.py"),
                        "-q", "-p", "no:cacheprovider", "-x"], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert " passed" in out
