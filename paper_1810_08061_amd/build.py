"""Build liblstm_dyn.so (the C ABI of include/lstm_dyn.h) for gfx950 with hipcc.

Each HIP source is compiled separately (in parallel) and linked into one
shared library next to this file.  Run: python -m paper_1810_08061_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "liblstm_dyn.so")
LIB_STRESS = os.path.join(HERE, "liblstm_dyn_stress.so")
SOURCES = ["api.hip", "prep.hip", "gemm.hip", "persistent.hip", "step.hip", "small.hip", "inproj.hip", "seq.hip", "pack.hip", "bwd.hip", "bwdblk.hip", "noalloc.hip"]
ARCH = "gfx950"
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.environ.get("HIPCC", f"{ROCM}/bin/hipcc")
# Packed fp32 instructions are disabled for all device code.
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
         "-Wno-unused-function", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str, build_dir: str = BUILD, extra=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False, stress: bool = False) -> str:
    """Build the library.  stress=True builds the timing-stress diagnostic
    variant instead (random sleeps before the loop kernel's stores of h, marks
    and polls), as liblstm_dyn_stress.so; the binding loads it when the
    environment variable LSTM_DYN_LIB names it."""
    build_dir = BUILD + ("_stress" if stress else "")
    lib = LIB_STRESS if stress else LIB
    extra = ("-DLDYN_STRESS=1",) if stress else ()
    os.makedirs(build_dir, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_dir, extra), SOURCES))
    tmp = lib + f".tmp{os.getpid()}"
    # rocBLAS (the backward pass's plain GEMMs) is not linked: the library
    # loads it with dlopen at the first forward for training
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp, "-ldl"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build(verbose=True, stress="--stress" in sys.argv)
    sys.exit(0)
