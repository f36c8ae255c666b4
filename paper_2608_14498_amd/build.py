"""Build the gfx950 HIP library in-tree: paper_2608_14498_amd/lib/librollplex.so.

    python -m paper_2608_14498_amd.build [-v] [--sanitize]

Every source is compiled by hipcc for gfx950 only.  Packed-fp32 instructions are
disabled for device code (-packed-fp32-ops); hipcc's host pass warns that it does
not know that feature, which is harmless.

--sanitize builds the same sources with AddressSanitizer and UndefinedBehaviorSanitizer
on the host code only (every -fsanitize= goes through -Xarch_host; device code is
unchanged) into _build/asan/librollplex.so, for the CPU tests of the host layer
(argument validation, workspace carving, the launch sequence up to the first HIP
call).  Load it with RP_LIBRARY=<path> and the ASan runtime preloaded.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "librollplex.so")
SOURCES = ["api.cpp", "elementwise.hip", "gemm.hip", "attention.hip", "calibrate.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out)


SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined"]
ASAN_LIB = os.path.join(ROOT, "_build", "asan", "librollplex.so")


def build(verbose: bool = False, sanitize: bool = False) -> str:
    objdir = os.path.join(ROOT, "_build", "asan" if sanitize else "")
    lib = ASAN_LIB if sanitize else LIB
    os.makedirs(os.path.dirname(lib), exist_ok=True)
    os.makedirs(objdir, exist_ok=True)
    extra = SANITIZE if sanitize else []
    objs = []
    jobs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src.replace(".", "_") + ".o")
        lang = ["-x", "hip"] if src.endswith(".cpp") else []
        jobs.append([HIPCC] + FLAGS + extra + lang + ["-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    with ThreadPoolExecutor(min(8, len(jobs))) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    tmp = lib + ".tmp"
    link = ["-Xarch_host", "-shared-libsan"] + extra if sanitize else []
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC"] + link + ["-o", tmp] + objs, verbose)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
