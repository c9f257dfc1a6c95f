"""Builds the HIP library libfno_spectral_conv.so for gfx950, in-tree.

    python -m paper_2307_15034_amd.build

Each source is compiled to an object in parallel (one hipcc per file) and the
objects are linked into one shared library next to this file, where the
Python binding loads it.  Every call rebuilds every object.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libfno_spectral_conv.so")
OBJ = os.path.join(HERE, "_build")
SOURCES = ["fno_kernels.hip", "fno_fast.hip", "fno_chain.hip", "fno_slab.hip", "fno_gemm.hip",
           "fno_wide.hip", "fno_wide2.hip", "fno_noalloc.hip", "fno_block.hip", "fno_plan.cpp"]
ARCH = "gfx950"


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
         # no packed-fp32 instructions anywhere in the device code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l)
    return res.returncode, errs


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ, exist_ok=True)
    objs, jobs = [], []
    for src in SOURCES:
        obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        jobs.append([hipcc()] + FLAGS + ["-I", os.path.join(ROOT, "include"), "-c",
                                         os.path.join(CSRC, src), "-o", obj])
    workers = max(1, min(len(jobs), os.cpu_count() or 1, 16))
    with cf.ThreadPoolExecutor(workers) as ex:
        results = list(ex.map(_run, jobs))
    for src, (rc, errs) in zip(SOURCES, results):
        if rc != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n" + errs)
        if verbose and errs.strip():
            print(errs, file=sys.stderr)
    rc, errs = _run([hipcc()] + FLAGS + ["-shared", "-o", LIB + ".tmp"] + objs)
    if rc != 0:
        raise RuntimeError("link failed:\n" + errs)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
