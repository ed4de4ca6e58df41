"""Builds the gfx950 shared library ``libaurora_delta.so`` in place.

    python -m paper_2602_11456_amd.build

Every call recompiles (a few seconds per source).  The library is built for
gfx950 only; hipcc cross-compiles it on a machine without a GPU.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB_NAME = "libaurora_delta.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-command-line-argument",
    # packed fp32 VALU forms are kept out of the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the ROCm toolchain is required to build")
    return path


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


PROBES = os.path.join(HERE, "probes")


def probe_sources():
    return sorted(glob.glob(os.path.join(PROBES, "*.hip")))


def build_probes(verbose: bool = False) -> list:
    """Compile every probes/*.hip (measurement executables the benchmark runs
    beside the library, e.g. the write ceilings of apply) into an executable
    of the same name; returns their paths."""
    out = []
    for src in probe_sources():
        exe = os.path.splitext(src)[0]
        tmp = exe + ".tmp"
        cmd = [hipcc(), *[f for f in HIPCC_FLAGS if f != "-fPIC"], src, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        os.replace(tmp, exe)
        out.append(exe)
    return out


def build(verbose: bool = False) -> str:
    """Compile every csrc/*.hip into one shared library (and the measurement
    probes); returns the library's path."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = []
    for src in sources():
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        cmd = [hipcc(), *HIPCC_FLAGS, "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        objs.append(obj)
    tmp = LIB_PATH + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB_PATH)
    build_probes(verbose)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
