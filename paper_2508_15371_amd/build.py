"""Build ``libcmsd.so`` (the gfx950 HIP kernels behind include/cmsd.h) in-tree.

Usage: ``python -m paper_2508_15371_amd.build [-v]``.  hipcc cross-compiles for
gfx950 on a host without a GPU.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "cmsd.hip")
INC = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libcmsd.so")

ARCH = "gfx950"
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared",
    # decisions and fixed summation orders rely on explicit fma() only
    "-ffp-contract=off",
    # packed fp32 VALU forms are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libcmsd.so)")


NATIVE_SRC = os.path.join(ROOT, "tests", "native", "logit_pass_native.cpp")
NATIVE_BIN = os.path.join(ROOT, "tests", "native", "logit_pass_native")


def build_native(verbose: bool = False) -> str:
    """Compile the native (C++, no Python) test consumer of libcmsd.so; returns its path."""
    cmd = [hipcc(), "-O2", "-std=c++17", "-I", INC, "-o", NATIVE_BIN, NATIVE_SRC, "-L", PKG, "-lcmsd",
           f"-Wl,-rpath,{PKG}", "-Wl,-rpath,$ORIGIN/../../paper_2508_15371_amd"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{r.stderr}")
    return NATIVE_BIN


PROBE_SRC = os.path.join(PKG, "csrc", "read_probe.hip")
PROBE_LIB = os.path.join(PKG, "libcmsd_readprobe.so")


def build_probe(verbose: bool = False) -> str:
    """Compile the benchmark's read-ceiling probe (a bare read of the same rows in the
    same grid shape as the joint row pass); returns its path."""
    tmp = PROBE_LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", *FLAGS, "-o", tmp, PROBE_SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{r.stderr}")
    os.replace(tmp, PROBE_LIB)
    return PROBE_LIB


def build(verbose: bool = False) -> str:
    """Compile libcmsd.so, then the native test consumer and the benchmark's read
    probe; returns the library's path.  Always recompiles."""
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", *FLAGS, "-I", INC, "-o", tmp, SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{r.stderr}")
    if verbose and err:
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    build_native(verbose)
    build_probe(verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
