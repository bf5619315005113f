"""Build the LAEP MoE C-ABI library (liblaep_moe.so) for gfx950 with hipcc.

Every HIP source is compiled for ``--offload-arch=gfx950`` only; the host
utility is plain C++.  The library is written next to this file so that it
travels with the source tree.  ``build()`` always recompiles.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "liblaep_moe.so")

HIP_SOURCES = ["route.hip", "route_bwd.hip", "counts.hip", "prune.hip", "compact.hip", "rowops.hip",
               "gemm_bf16.hip", "gemm_bwd.hip", "gemm_f32.hip", "calib.hip"]
HIP_HOST_SOURCES = ["api.cpp", "streams.cpp"]   # host code that calls the HIP runtime
CXX_SOURCES = ["rearrange.cpp"]         # plain host C++

ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          "-Wno-unused-variable", "-Wno-unused-but-set-variable"]
# The packed-fp32 feature is disabled for device code (hipcc's host pass
# reports it as unknown, which is harmless).
HIP_FLAGS = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang",
             "-packed-fp32-ops"]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build liblaep_moe.so)")


def _compile(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops" not in l and "is not a recognized feature" not in l)
    return r.returncode, " ".join(cmd), out


def build(verbose: bool = False) -> str:
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    jobs, objs = [], []
    for src in HIP_SOURCES + HIP_HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        objs.append(obj)
        lang = ["-x", "hip"]
        jobs.append([hipcc, *lang, *COMMON, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
    for src in CXX_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        objs.append(obj)
        jobs.append(["g++", *COMMON, "-c", os.path.join(CSRC, src), "-o", obj])
    n_workers = min(len(jobs), max(1, min(8, os.cpu_count() or 1)))
    with concurrent.futures.ThreadPoolExecutor(n_workers) as ex:
        results = list(ex.map(_compile, jobs))
    failed = False
    for rc, cmd, out in results:
        if verbose or rc != 0:
            print(cmd)
            if out.strip():
                print(out)
        failed |= rc != 0
    if failed:
        raise RuntimeError("liblaep_moe.so: compilation failed")
    tmp = LIB + ".tmp"
    rc, cmd, out = _compile([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    if rc != 0:
        print(cmd)
        print(out)
        raise RuntimeError("liblaep_moe.so: link failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
