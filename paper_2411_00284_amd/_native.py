"""ctypes loader for ``libfsdp_bucket.so`` (the C ABI of ``include/fsdp_bucket.h``).

torch is imported first so that the library binds to the HIP runtime torch
already loaded (both carry the soname ``libamdhip64.so.7``): device pointers
and the ``hipStream_t`` handles torch hands out are then valid in the
library.  Loading fails loudly when the library has not been built; there is
no fallback.
"""

from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (must precede the library: shared HIP runtime)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfsdp_bucket.so")

c_status = ctypes.c_int32
c_plan_p = ctypes.c_void_p
c_ptr_array = ctypes.POINTER(ctypes.c_void_p)

# name -> (restype, argtypes); mirrors include/fsdp_bucket.h
SIGNATURES = {
    "fsdp_bucket_plan": (c_status, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
                                    ctypes.POINTER(ctypes.c_int64), ctypes.c_int32,
                                    ctypes.POINTER(ctypes.c_void_p)]),
    "fsdp_bucket_plan_ex": (c_status, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
                                       ctypes.POINTER(ctypes.c_int64), ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.POINTER(ctypes.c_void_p)]),
    "fsdp_plan_free": (None, [c_plan_p]),
    "fsdp_plan_chunk_elems": (ctypes.c_int64, [c_plan_p]),
    "fsdp_plan_world_size": (ctypes.c_int32, [c_plan_p]),
    "fsdp_plan_num_params": (ctypes.c_int32, [c_plan_p]),
    "fsdp_plan_param": (c_status, [c_plan_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
                                   ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]),
    "fsdp_plan_local_rows": (ctypes.c_int64, [c_plan_p, ctypes.c_int32, ctypes.c_int32]),
    "fsdp_status_str": (ctypes.c_char_p, [c_status]),
    "fsdp_last_error": (ctypes.c_char_p, []),
    "fsdp_ag_pack": (c_status, [c_plan_p, ctypes.c_int32, c_ptr_array, ctypes.c_void_p, ctypes.c_void_p]),
    "fsdp_ag_unpack": (c_status, [c_plan_p, ctypes.c_void_p, c_ptr_array, ctypes.c_void_p]),
    "fsdp_rs_pack": (c_status, [c_plan_p, c_ptr_array, ctypes.c_void_p, ctypes.c_void_p]),
    "fsdp_rs_reduce": (c_status, [c_plan_p, ctypes.c_int32, ctypes.c_void_p, c_ptr_array, ctypes.c_void_p]),
    "fsdp_ag_pack_ex": (c_status, [c_plan_p, ctypes.c_int32, c_ptr_array, ctypes.c_int32, ctypes.c_void_p,
                                   ctypes.c_void_p]),
    "fsdp_ag_pack_push": (c_status, [c_plan_p, ctypes.c_int32, c_ptr_array, ctypes.c_int32, c_ptr_array,
                                     ctypes.c_void_p]),
    "fsdp_ag_unpack_ex": (c_status, [c_plan_p, ctypes.c_int32, c_ptr_array, c_ptr_array, ctypes.c_void_p]),
    "fsdp_rs_pack_ex": (c_status, [c_plan_p, ctypes.c_int32, c_ptr_array, ctypes.c_int32, c_ptr_array,
                                   ctypes.c_void_p]),
    "fsdp_rs_reduce_ex": (c_status, [c_plan_p, ctypes.c_int32, ctypes.c_int32, c_ptr_array, c_ptr_array,
                                     ctypes.c_void_p]),
    "fsdp_auto_wrap": (c_status, [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(ctypes.c_int64), ctypes.c_double, ctypes.c_double,
                                  ctypes.c_double, ctypes.c_double, ctypes.c_int64,
                                  ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)]),
}

class PlanOptions(ctypes.Structure):
    """struct fsdp_plan_options."""
    _fields_ = [("max_workgroups", ctypes.c_int64), ("reduce_tiles", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


REDUCE_TILES = {"auto": 0, "full": 1, "half": 2}
MAX_PARAMS = 64
MAX_CHUNKS = 128
DTYPE_BF16 = 0
DTYPE_F32 = 1
DTYPE_F16 = 2

_lib = None


def _hip_runtimes_mapped() -> set[str]:
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    paths.add(os.path.realpath(line.split()[-1]))
    except OSError:
        pass
    return paths


def load() -> ctypes.CDLL:
    """Load the library once; raises if it is missing or binds a second HIP runtime."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built: run `python -m paper_2411_00284_amd.build` "
            "first; there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise ImportError(f"two HIP runtimes are mapped ({sorted(runtimes)}); "
                          "import torch before loading libfsdp_bucket.so")
    _lib = lib
    return lib
