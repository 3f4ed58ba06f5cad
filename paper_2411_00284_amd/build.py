"""Build the gfx950 shared library ``libfsdp_bucket.so`` in-tree.

Runs on a machine without a GPU (hipcc cross-compiles for gfx950).  The
kernels are built without fast-math and without fp contraction, and with the
packed-fp32 target feature turned off, so the compiler emits only scalar fp32
adds and the correctly rounded fp32 division sequence.

Usage: ``python -m paper_2411_00284_amd.build`` (or ``build()`` from Python).
``-DNAME=VALUE`` overrides a tuning macro (``FSDP_PACK_BLOCK``,
``FSDP_BLOCKS_PER_CU``, ...) and ``--out DIR`` writes that variant's library
to DIR instead of the package (the benchmark's ``--library`` loads it), for
measuring launch shapes; results never depend on them.
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


def build(verbose: bool = False, defines=(), out_dir: str | None = None) -> str:
    """Compile every source and link the library; returns its path.  With
    ``defines`` (``NAME=VALUE`` macro overrides) or ``out_dir``, only the
    bucket library is built, into ``out_dir``."""
    variant = bool(defines) or out_dir is not None
    bdir = os.path.join(out_dir, "_build") if out_dir else BUILD
    lib_path = os.path.join(out_dir, LIB_NAME) if out_dir else LIB_PATH
    os.makedirs(bdir, exist_ok=True)
    inc = [f"-I{INCLUDE}", f"-I{CSRC}", f"-I{os.path.join(ROCM, 'include')}"]
    dflags = [f"-D{d}" for d in defines]
    kobj = os.path.join(bdir, "bucket_kernels.o")
    _run([HIPCC, *DEVICE_FLAGS, *dflags, *inc, "-c", os.path.join(CSRC, "bucket_kernels.hip"), "-o", kobj], verbose)
    hobjs = []
    for src in HOST_SOURCES:
        obj = os.path.join(bdir, os.path.splitext(src)[0] + ".o")
        _run(["g++", *HOST_FLAGS, *dflags, *inc, "-c", os.path.join(CSRC, src), "-o", obj], verbose)
        hobjs.append(obj)
    tmp = lib_path + f".tmp{os.getpid()}"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, kobj, *hobjs], verbose)
    os.replace(tmp, lib_path)
    if variant:
        return lib_path
    pobj = os.path.join(BUILD, "ceiling_probes.o")
    _run([HIPCC, *DEVICE_FLAGS, *inc, "-c", os.path.join(CSRC, "ceiling_probes.hip"), "-o", pobj], verbose)
    tmp = PROBES_PATH + f".tmp{os.getpid()}"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, pobj], verbose)
    os.replace(tmp, PROBES_PATH)
    return LIB_PATH


def clean() -> None:
    shutil.rmtree(BUILD, ignore_errors=True)


if __name__ == "__main__":
    args = sys.argv[1:]
    defs = [a[2:] for a in args if a.startswith("-D")]
    out = args[args.index("--out") + 1] if "--out" in args else None
    print(build(verbose="-v" in args, defines=defs, out_dir=out))
