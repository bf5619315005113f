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
               "gemm_bf16.hip", "gemm_bwd.hip", "gemm_f32.hip", "calib.hip", "noalloc.hip"]
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


# ---------------------------------------------------------------------------
# Host sanitizer build (CPU checking only; never loaded by the product path).
# The host-only sources (argument validation, workspace sizing, the side
# streams, the rearrangement utility) are compiled with clang's address and
# undefined-behaviour sanitizers and linked with the ordinary HIP objects of
# build(), whose device code is untouched.  tests/test_host_sanitizers.py runs
# the C-ABI contract tests against the result with the sanitizer runtime
# preloaded.
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
             "-fno-omit-frame-pointer", "-g", "-O1"]


def _clangxx() -> str:
    for cand in ("/opt/rocm/llvm/bin/clang++", shutil.which("clang++")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("clang++ not found (needed for the host sanitizer build)")


def sanitizer_runtime() -> str:
    """Path of clang's shared address-sanitizer runtime (to preload)."""
    cxx = _clangxx()
    r = subprocess.run([cxx, "-print-file-name=libclang_rt.asan-x86_64.so"],
                       stdout=subprocess.PIPE, text=True, check=True)
    path = r.stdout.strip()
    if not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError("clang's shared ASan runtime was not found")
    return path


def build_host_sanitized(out_dir: str, verbose: bool = False) -> str:
    """liblaep_moe_hostsan.so in out_dir: host sources under ASan + UBSan,
    HIP objects as build() made them (built first when missing)."""
    cxx = _clangxx()
    os.makedirs(out_dir, exist_ok=True)
    hip_objs = [os.path.join(BUILD, src + ".o") for src in HIP_SOURCES]
    if not all(os.path.exists(o) for o in hip_objs):
        build(verbose=verbose)
    inc = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]
    jobs, san_objs = [], []
    for src in HIP_HOST_SOURCES + CXX_SOURCES:
        obj = os.path.join(out_dir, src + ".san.o")
        san_objs.append(obj)
        jobs.append([cxx, "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function", *SAN_FLAGS,
                     *inc, "-c", os.path.join(CSRC, src), "-o", obj])
    with concurrent.futures.ThreadPoolExecutor(len(jobs)) as ex:
        results = list(ex.map(_compile, jobs))
    for rc, cmd, out in results:
        if verbose or rc != 0:
            print(cmd)
            print(out)
        if rc != 0:
            raise RuntimeError("host sanitizer build: compilation failed")
    lib_out = os.path.join(out_dir, "liblaep_moe_hostsan.so")
    rc, cmd, out = _compile([cxx, "-shared", "-fPIC", *SAN_FLAGS, "-shared-libasan", *san_objs,
                             *hip_objs, "-L/opt/rocm/lib", "-lamdhip64",
                             "-Wl,-rpath,/opt/rocm/lib", "-o", lib_out])
    if rc != 0:
        print(cmd)
        print(out)
        raise RuntimeError("host sanitizer build: link failed")
    return lib_out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
