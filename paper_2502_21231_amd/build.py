"""Builds libbs_attn.so (HIP for gfx950) in-tree with hipcc, and libbs_hdp.so (host-only
planners) with the host C++ compiler.

    python -m paper_2502_21231_amd.build [-v]

Every source is compiled on every call (the build check must really compile);
objects go to paper_2502_21231_amd/_build/, the libraries to
paper_2502_21231_amd/libbs_attn.so and paper_2502_21231_amd/libbs_hdp.so.
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
LIB = os.path.join(PKG, "libbs_attn.so")

SOURCES = ["plan.hip", "fwd_bf16.hip", "dq_bf16.hip", "dkdv_bf16.hip", "f32.hip", "rowwise.hip",
           "xent.hip", "capi.hip"]
# per-source additions: the dQ kernel's loop schedules faster under the backend's max-ILP
# strategy (the forward's and dK/dV's do not)
SOURCE_FLAGS = {"dq_bf16.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"]}
# host-only planners (no GPU code): a library of their own, built with the host compiler
HDP_SOURCE = "hdp.cpp"
HDP_LIB = os.path.join(PKG, "libbs_hdp.so")
HDP_CFLAGS = ["-O2", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off", "-Wall", "-Wextra"]

ARCH = "gfx950"
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-munsafe-fp-atomics",
    # hipcc forms packed-fp32 instructions by itself from scalar float code;
    # keep them out of the device code (the host pass warns it does not know the
    # feature, which is harmless)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP toolchain is required to build libbs_attn.so")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def host_cxx() -> str:
    for cand in (shutil.which("g++"), shutil.which("c++"), shutil.which("clang++")):
        if cand:
            return cand
    raise RuntimeError("no host C++ compiler found (g++) to build libbs_hdp.so")


def build_hdp(verbose: bool = False) -> str:
    """Compiles the host planners into libbs_hdp.so; returns its path."""
    tmp = HDP_LIB + ".tmp"
    _run([host_cxx(), *HDP_CFLAGS, os.path.join(CSRC, HDP_SOURCE), "-o", tmp], verbose)
    os.replace(tmp, HDP_LIB)
    return HDP_LIB


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compiles all HIP sources for gfx950 and links libbs_attn.so, and builds the host planners'
    libbs_hdp.so; returns the path of libbs_attn.so."""
    build_hdp(verbose)
    cc = hipcc()
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmds.append([cc, *CFLAGS, *SOURCE_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj])
    jobs = jobs or min(len(cmds), max(1, min(8, os.cpu_count() or 1)))
    with ThreadPoolExecutor(jobs) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
