"""Builds libpss.so (the layer's HIP sources, gfx950) and libpss_bench.so
(the measurement kernels) in place, next to this file.

Usage:  python -m paper_2207_10731_amd.build   (or build() from Python)
Each source is compiled in its own hipcc process, then linked; the library is
written to a temporary name and renamed, so a reader never sees a half-built
file.  Packed-fp32 instruction selection is switched off for device code.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libpss.so")
SOURCES = ["pss_api.hip", "pss_forward.hip", "pss_backward.hip", "pss_sorted.hip",
           "pss_sparse.hip", "pss_addr.hip"]
BENCH_LIB = os.path.join(PKG, "libpss_bench.so")
BENCH_SOURCES = ["pss_bench.hip"]
ARCH = "gfx950"

CXXFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-munsafe-fp-atomics",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    cand = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    return cand if os.path.exists(cand) else (shutil.which("hipcc") or "hipcc")


def _run(cmd):
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if res.returncode != 0:
        raise RuntimeError("build step failed:\n" + " ".join(cmd) + "\n" + res.stdout)
    return res.stdout


def _link(objs, lib):
    tmp = lib + ".tmp"
    out = _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, lib)
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    cmds = []
    objs = {}
    for src in SOURCES + BENCH_SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        objs[src] = obj
        cmds.append([hipcc(), *CXXFLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
    with ThreadPoolExecutor(max_workers=min(len(cmds), 4)) as ex:
        outs = list(ex.map(_run, cmds))
    outs.append(_link([objs[s] for s in SOURCES], LIB))
    outs.append(_link([objs[s] for s in BENCH_SOURCES], BENCH_LIB))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
