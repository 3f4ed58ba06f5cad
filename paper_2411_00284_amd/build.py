"""Build the gfx950 shared library ``libfsdp_bucket.so`` in-tree.

Runs on a machine without a GPU (hipcc cross-compiles for gfx950).  The
kernels are built without fast-math and without fp contraction, and with the
packed-fp32 target feature turned off, so the compiler emits only scalar fp32
adds and the correctly rounded fp32 division sequence.

Usage: ``python -m paper_2411_00284_amd.build`` (or ``build()`` from Python).
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB_NAME = "libfsdp_bucket.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
# Reference streams for the benchmark's ceiling leg: a library of their own,
# not loaded by the package.
PROBES_PATH = os.path.join(PKG, "libfsdp_probes.so")

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

DEVICE_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]
HOST_SOURCES = ["plan.cpp", "auto_wrap.cpp"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-ffp-contract=off", "-D__HIP_PLATFORM_AMD__"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"build step failed ({res.returncode}): {' '.join(cmd)}\n{res.stdout}\n{res.stderr}")
    return res


def build(verbose: bool = False) -> str:
    """Compile every source and link the library; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    inc = [f"-I{INCLUDE}", f"-I{CSRC}", f"-I{os.path.join(ROCM, 'include')}"]
    kobj = os.path.join(BUILD, "bucket_kernels.o")
    _run([HIPCC, *DEVICE_FLAGS, *inc, "-c", os.path.join(CSRC, "bucket_kernels.hip"), "-o", kobj], verbose)
    hobjs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        _run(["g++", *HOST_FLAGS, *inc, "-c", os.path.join(CSRC, src), "-o", obj], verbose)
        hobjs.append(obj)
    tmp = LIB_PATH + f".tmp{os.getpid()}"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, kobj, *hobjs], verbose)
    os.replace(tmp, LIB_PATH)
    pobj = os.path.join(BUILD, "ceiling_probes.o")
    _run([HIPCC, *DEVICE_FLAGS, *inc, "-c", os.path.join(CSRC, "ceiling_probes.hip"), "-o", pobj], verbose)
    tmp = PROBES_PATH + f".tmp{os.getpid()}"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, pobj], verbose)
    os.replace(tmp, PROBES_PATH)
    return LIB_PATH


def clean() -> None:
    shutil.rmtree(BUILD, ignore_errors=True)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
