"""Build the gfx950 library in-tree.

1. compile and run the table generator (host C++) -> csrc/generated/mace_tables.h
   (FP32 immediates) and mace_tables64.h (FP64, for the debug precision)
2. compile the host neighbour list with g++ (-ffp-contract=off: its FP64
   arithmetic must round exactly as written)
3. hipcc every kernel file and the host runtime for gfx950 -> libmace_amd.so
   (the device neighbour list with -ffp-contract=off, like the host one)
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmace_amd.so")
HIP_SOURCES = ["api.hip", "k_edge.hip", "k_radial.hip", "k_tpr.hip", "k_layer0.hip", "k_sender.hip", "k_symcon.hip", "k_node.hip",
               "k_neighbors.hip", "k_fp64.hip"]
# files whose FP64 arithmetic must round exactly as written (no fused multiply-adds)
NO_CONTRACT = {"k_neighbors.hip"}
HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-Wall", "-Wno-unused-function",
    "-Wno-unused-variable", "-Wno-unused-but-set-variable",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout)
        raise RuntimeError(f"build step failed: {' '.join(cmd[:3])} ...")
    return r.stdout


def build(verbose: bool = False, jobs: int = 8) -> str:
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(os.path.join(CSRC, "generated"), exist_ok=True)
    gen = os.path.join(BUILD, "gen_tables")
    _run(["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-o", gen, os.path.join(CSRC, "gen_tables.cpp")], verbose)
    _run([gen, os.path.join(CSRC, "generated", "mace_tables.h"), os.path.join(CSRC, "generated", "mace_tables64.h")],
         verbose)
    nl_obj = os.path.join(BUILD, "neighbors.o")
    _run(["g++", "-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-Wno-unknown-pragmas", "-c",
          os.path.join(CSRC, "neighbors.cpp"), "-o", nl_obj], verbose)
    objs = []
    procs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        extra = ["-ffp-contract=off"] if src in NO_CONTRACT else []
        cmd = [hipcc] + HIPCC_FLAGS + extra + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
        objs.append(obj)
        if len([p for p in procs if p[1].poll() is None]) >= jobs:
            procs[0][1].wait()
    failed = []
    for cmd, p in procs:
        out, _ = p.communicate()
        if p.returncode != 0:
            failed.append(out)
        elif verbose and out.strip():
            print(out)
    if failed:
        sys.stderr.write("\n".join(failed))
        raise RuntimeError("hipcc failed")
    tmp = LIB + ".tmp"
    _run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp] + objs + [nl_obj], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
