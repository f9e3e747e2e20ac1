"""Builds libembx.so (HIP kernels for gfx950 + the C ABI + the host planner) in-tree.

    python paper_2507_01676_amd/build.py
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libembx.so")
ARCH = "gfx950"

HIP_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-ffp-contract=off",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", os.path.join(ROOT, "include")]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-fast-math", "-Wall"]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd[:3])} ...")
    return r


# lookup.hip is compiled in parts (EMBX_PART): one per (row type, weighted) kernel
# family, plus the probes, filler and launch code
LOOKUP_PARTS = 5
# gather.hip: one part per (row type, weighted) kernel family, each built for every number
# of row loads in flight per step a plan may choose (kGatherStepChoices in device_types.hpp)
GATHER_PARTS = 4
GATHER_STEPS = (12, 13, 16)


def _run_all(cmds, verbose):
    """Runs the compile commands in parallel; raises on the first failure."""
    procs = []
    for cmd in cmds:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    failed = None
    for cmd, p in procs:
        out, _ = p.communicate()
        if p.returncode != 0 and failed is None:
            failed = (cmd, out)
    if failed is not None:
        sys.stderr.write(failed[1])
        raise RuntimeError(f"build step failed: {' '.join(failed[0][:3])} ...")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    cmds, objs = [], []
    for part in range(LOOKUP_PARTS):
        o = os.path.join(BUILD, f"lookup_{part}.o")
        cmds.append([hipcc, *HIP_FLAGS, f"-DEMBX_PART={part}", "-c", os.path.join(CSRC, "lookup.hip"), "-o", o])
        objs.append(o)
    for ks in GATHER_STEPS:
        for part in range(GATHER_PARTS):
            o = os.path.join(BUILD, f"gather_{part}_k{ks}.o")
            cmds.append([hipcc, *HIP_FLAGS, f"-DEMBX_GPART={part}", f"-DEMBX_GKS={ks}", "-c",
                         os.path.join(CSRC, "gather.hip"), "-o", o])
            objs.append(o)
    o = os.path.join(BUILD, "api.o")
    cmds.append([hipcc, *HIP_FLAGS, "-x", "hip", "-c", os.path.join(CSRC, "api.cpp"), "-o", o])
    objs.append(o)
    # the planner is plain host C++: every binary64 operation rounds as written
    o = os.path.join(BUILD, "planner.o")
    cmds.append(["g++", *HOST_FLAGS, "-c", os.path.join(CSRC, "planner.cpp"), "-o", o])
    objs.append(o)
    _run_all(cmds, verbose)
    tmp = LIB + ".tmp"
    _run([hipcc, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
