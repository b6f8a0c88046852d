"""Build libff.so (the HIP kernels and the C ABI of include/ff.h) for gfx950.

Run ``python -m paper_2609_14706_amd.build`` (or call :func:`build`).  The
library is written next to this file and loaded from there by the binding.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libff.so")
BENCH = os.path.join(HERE, "ffbench")
SOURCES = ["ff_gemm_bf16.hip", "ff_gemm_f32.hip", "ff_chol.hip", "ff_aux.hip", "ff_waterkron.hip",
           "ff_engine.hip"]
ARCH = "gfx950"
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-result", f"-I{INCLUDE}", f"-I{CSRC}"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    cc = hipcc()
    objdir = os.path.join(ROOT, "_build")
    os.makedirs(objdir, exist_ok=True)

    def compile_one(src):
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        cmd = [cc, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"compiling {src} failed:\n{r.stdout}\n{r.stderr}")
        if verbose:
            print("compiled", src, flush=True)
        return obj

    with ThreadPoolExecutor(min(len(SOURCES), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking libff.so failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB, flush=True)
    return LIB


def build_bench(verbose: bool = False) -> bool:
    """Build the native measurement driver of the C ABI (ffbench, used for
    hardware-counter runs) against the built library.  Separate from the
    library build: a failure here is reported and returns False."""
    cmd = [hipcc(), *FLAGS, os.path.join(CSRC, "ffbench.hip"), "-o", BENCH + ".tmp",
           f"-L{HERE}", "-lff", "-Wl,-rpath,$ORIGIN"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        print(f"building ffbench failed (the library is unaffected):\n{r.stdout}\n{r.stderr}",
              file=sys.stderr, flush=True)
        return False
    os.replace(BENCH + ".tmp", BENCH)
    if verbose:
        print("built", BENCH, flush=True)
    return True


if __name__ == "__main__":
    build(verbose=True)
    build_bench(verbose=True)
    sys.exit(0)
