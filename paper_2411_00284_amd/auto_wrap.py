"""Binding of ``fsdp_auto_wrap``: SimpleFSDP's auto-wrapping decision
(section 3.3.2, Algorithm 1, Table 1), computed by the library's host code.

Argument marshalling only: the node tables are copied into C arrays, the
library cuts them into buckets, and the bucket numbers come back as lists of
node indices.
"""

from __future__ import annotations

import ctypes
from typing import Sequence

from . import _native
from .bucket import _check

__all__ = ["auto_wrap"]


def _arr(ctype, values, n, what):
    if len(values) != n:
        raise ValueError(f"{what}: expected {n} entries, got {len(values)}")
    return (ctype * max(n, 1))(*values)


def auto_wrap(ag_words: Sequence[int], compute_time: Sequence[float], compute_mem: Sequence[int],
              alpha_ag: float, beta_ag: float, mem_max: int, backward: bool = False,
              rs_words: Sequence[int] | None = None, alpha_rs: float = 0.0,
              beta_rs: float = 0.0) -> list[list[int]]:
    """Cut one pass's all-gather nodes (in the order the pass computes them)
    into consecutive buckets; returns the buckets as lists of node indices.

    ``ag_words[i]``, ``compute_time[i]`` and ``compute_mem[i]`` are node i's
    all-gather words, compute time and peak compute memory; ``rs_words`` (the
    backward pass only) its gradient's reduce-scatter words.  A collective
    moving n words costs ``alpha + beta * n``; ``mem_max`` bounds a bucket's
    summed memory.
    """
    lib = _native.load()
    n = len(ag_words)
    ag = _arr(ctypes.c_int64, [int(x) for x in ag_words], n, "ag_words")
    t = _arr(ctypes.c_double, [float(x) for x in compute_time], n, "compute_time")
    m = _arr(ctypes.c_int64, [int(x) for x in compute_mem], n, "compute_mem")
    rs = None
    if backward:
        if rs_words is None:
            raise ValueError("rs_words is required for a backward pass")
        rs = _arr(ctypes.c_int64, [int(x) for x in rs_words], n, "rs_words")
    out = (ctypes.c_int32 * max(n, 1))()
    nb = ctypes.c_int32(-1)
    _check(lib.fsdp_auto_wrap(n, 1 if backward else 0, ag, rs, t, m, float(alpha_ag), float(beta_ag),
                              float(alpha_rs), float(beta_rs), int(mem_max), out, ctypes.byref(nb)),
           "fsdp_auto_wrap")
    buckets: list[list[int]] = [[] for _ in range(nb.value)]
    for i in range(n):
        buckets[out[i]].append(i)
    return buckets
