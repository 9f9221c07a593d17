"""Build libatom.so in-tree for gfx950 with hipcc.

Usage: python -m paper_2403_10504_amd.build [-v] [--changed]

Every source is compiled on each call (the build check compiles from
scratch); --changed recompiles only the objects older than their source or
any header of csrc/ or include/ (a developer's rebuild).  HIP sources get `-Xclang -target-feature -Xclang -packed-fp32-ops`
so the compiler never emits packed fp32 arithmetic; the host pass warns that
it does not know the feature, which is harmless.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libatom.so")
ARCH = "gfx950"

HIP_SOURCES = ["gemm.hip", "attention.hip", "attention_f32.hip", "rowops.hip", "runtime.cpp", "nodes.cpp", "schedule.cpp",
               "host_accum.cpp", "transfer.cpp", "capi_kernels.cpp"]
# per-source optimisation level (see attention_f32.hip)
OPT = {"attention_f32.hip": "-O1"}
CXX_SOURCES = ["plan.cpp"]


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libatom)")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def _stale(src, obj):
    if not os.path.exists(obj):
        return True
    t = os.path.getmtime(obj)
    deps = [os.path.join(CSRC, src)]
    deps += [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")]
    inc = os.path.join(os.path.dirname(HERE), "include")
    deps += [os.path.join(inc, f) for f in os.listdir(inc) if f.endswith(".h")]
    return any(os.path.getmtime(p) > t for p in deps)


def build(verbose: bool = False, jobs: int | None = None, changed_only: bool = False) -> str:
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    common = ["-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function", "-I", CSRC]
    # extra compiler flags, e.g. a -D override of a tile configuration
    common += os.environ.get("ATOM_HIPCC_FLAGS", "").split()
    cmds, objs = [], []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        cmds.append([hipcc, f"--offload-arch={ARCH}", "-x", "hip", OPT.get(src, "-O3"), *common,
                     "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                     "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
        if changed_only and not _stale(src, obj):
            cmds.pop()
    for src in CXX_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        cmds.append(["g++", "-O3", *common, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
        if changed_only and not _stale(src, obj):
            cmds.pop()
    jobs = jobs or max(1, min(8, len(cmds)))
    with ThreadPoolExecutor(jobs) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-o", tmp, *objs, "-lhsa-runtime64", "-lpthread"], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, changed_only="--changed" in sys.argv))
