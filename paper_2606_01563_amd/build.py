"""Build libmomentkv.so in-tree with hipcc for gfx950.

    python -m paper_2606_01563_amd.build        # or __graft_entry__.build()

Sources: csrc/*.hip (kernels) and csrc/*.cpp (C ABI), compiled in parallel to
objects under csrc/_build/ and linked into paper_2606_01563_amd/libmomentkv.so.
Always recompiles (a cheap, explicit "does it build" step).
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(CSRC, "_build")
LIB = os.path.join(PKG, "libmomentkv.so")
ROOT = os.path.dirname(PKG)

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 vector instructions are disabled for all device code.
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-variable", "-Wno-unused-function",
          f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]


# Host-side AddressSanitizer and UndefinedBehaviorSanitizer for the sanitized copy of the
# library (each -fsanitize= applies to the host pass only; device code is built as usual).
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all",
            "-shared-libasan"]
OBJ_SAN = os.path.join(CSRC, "_build_san")
LIB_SAN = os.path.join(OBJ_SAN, "libmomentkv_san.so")


def _compile(src: str, sanitize: bool = False) -> tuple[str, int, str]:
    obj = os.path.join(OBJ_SAN if sanitize else OBJ, os.path.basename(src) + ".o")
    cmd = [HIPCC, *COMMON, *(SANITIZE if sanitize else []), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    return obj, r.returncode, out


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compile and link the library; sanitize=True builds the host-sanitized copy
    (csrc/_build_san/libmomentkv_san.so, for the CPU-only checks of the C ABI's validation
    code) and leaves the product library alone."""
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(OBJ_SAN if sanitize else OBJ, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    jobs = min(len(srcs), max(1, min(16, os.cpu_count() or 1)))
    with ThreadPoolExecutor(jobs) as ex:
        results = list(ex.map(lambda x: _compile(x, sanitize), srcs))
    failed = [(o, out) for o, rc, out in results if rc != 0]
    for o, rc, out in results:
        if out.strip() and (verbose or rc != 0):
            print(out, file=sys.stderr)
    if failed:
        raise RuntimeError("hipcc failed for: " + ", ".join(os.path.basename(o) for o, _ in failed))
    lib = LIB_SAN if sanitize else LIB
    tmp = lib + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *(SANITIZE if sanitize else []),
           *[o for o, _, _ in results], "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        print(r.stdout + r.stderr, file=sys.stderr)
        raise RuntimeError("link failed")
    shutil.move(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
