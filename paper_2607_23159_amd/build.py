"""Build the gfx950 shared library ``libcachedsearch.so`` in-tree.

Each ``csrc/*.hip`` file is compiled to an object with hipcc for gfx950 (in
parallel), then linked into one shared library next to this file.  Packed
fp32 VALU instructions are disabled for all device code.

Usage: ``python -m paper_2607_23159_amd.build`` (or ``build()``).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libcachedsearch.so")
ARCH = "gfx950"


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-result", "-Wno-unused-value", "-I", os.path.join(ROOT, "include")]


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.basename(src) + ".o")
    cmd = [hipcc()] + FLAGS + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(OBJ, exist_ok=True)
    srcs = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}"] + objs + ["-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} from {len(srcs)} sources", file=sys.stderr)
    return LIB


# Host-side sanitizer build of the C ABI (AddressSanitizer + UBSan on the
# host code only; device code is compiled as usual) linked with the ABI check
# driver tests/abi_check.cpp, which exercises the ranking call and every entry
# point's argument validation without a GPU.
SAN_DIR = os.path.join(OBJ, "asan")
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]


def _stale(target: str, deps) -> bool:
    if not os.path.exists(target):
        return True
    t = os.path.getmtime(target)
    return any(os.path.getmtime(d) > t for d in deps)


def build_abi_check() -> str:
    """Build (when a source changed) and return the path of the sanitized
    ABI check executable."""
    os.makedirs(SAN_DIR, exist_ok=True)
    inc = os.path.join(ROOT, "include")
    hdrs = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hpp", ".h"))] + \
        [os.path.join(inc, "cs.h")]
    srcs = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))
    flags = ["-O1", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Xclang", "-target-feature",
             "-Xclang", "-packed-fp32-ops", "-Wno-unused-result", "-Wno-unused-value", "-I", inc] + SAN_HOST

    def one(src):
        obj = os.path.join(SAN_DIR, os.path.basename(src) + ".o")
        if _stale(obj, [src] + hdrs):
            r = subprocess.run([hipcc()] + flags + ["-c", src, "-o", obj], capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"sanitized compile of {src} failed:\n{r.stderr}")
        return obj

    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(one, srcs))
    drv = os.path.join(ROOT, "tests", "abi_check.cpp")
    drv_o = os.path.join(SAN_DIR, "abi_check.o")
    clangxx = os.path.join(os.path.dirname(hipcc()), "..", "llvm", "bin", "clang++")
    if _stale(drv_o, [drv, os.path.join(inc, "cs.h")]):
        r = subprocess.run([clangxx, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined",
                            "-fno-omit-frame-pointer", "-I", inc, "-c", drv, "-o", drv_o],
                           capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"compile of {drv} failed:\n{r.stderr}")
    exe = os.path.join(SAN_DIR, "abi_check")
    if _stale(exe, objs + [drv_o]):
        r = subprocess.run([hipcc(), f"--offload-arch={ARCH}"] + SAN_HOST[:4] + objs + [drv_o, "-o", exe],
                           capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link of {exe} failed:\n{r.stderr}")
    return exe


if __name__ == "__main__":
    build()
