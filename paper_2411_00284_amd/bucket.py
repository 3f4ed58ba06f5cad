"""Thin Python binding over the C ABI (argument marshalling only).

Every step of the path runs in the HIP kernels of ``libfsdp_bucket.so``;
this module only turns torch tensors into device pointers, checks that their
dtype, device and element count match the plan, and raises on a non-zero
status.  torch provides device memory and the current HIP stream.
"""

from __future__ import annotations

import ctypes
import math
from typing import Sequence

import torch

from . import _native

BF16_DTYPES = (torch.bfloat16, torch.int16, torch.uint16)
F16_DTYPES = (torch.float16,)
F32_DTYPES = (torch.float32, torch.int32)
_DTYPE_CODES = {"bf16": 0, "f32": 1, "f16": 2}
_DTYPES = {"bf16": BF16_DTYPES, "f16": F16_DTYPES, "f32": F32_DTYPES}


def _dtype_code(name: str) -> int:
    if name not in _DTYPE_CODES:
        raise ValueError("dtype must be 'bf16', 'f16' or 'f32'")
    return _DTYPE_CODES[name]


def _elem_dtypes(name: str):
    _dtype_code(name)
    return _DTYPES[name]


def _dtype_name(t: torch.Tensor) -> str:
    for name, dtypes in _DTYPES.items():
        if t.dtype in dtypes:
            return name
    raise TypeError(f"unsupported dtype {t.dtype}")


class FsdpError(RuntimeError):
    """A non-zero status from the library."""

    def __init__(self, status: int, where: str):
        lib = _native.load()
        msg = lib.fsdp_status_str(status).decode()
        detail = lib.fsdp_last_error().decode()
        super().__init__(f"{where}: {msg}" + (f" ({detail})" if detail else ""))
        self.status = status


def _check(status: int, where: str) -> None:
    if status != 0:
        raise FsdpError(status, where)


def _rows_inner(shape) -> tuple[int, int]:
    shape = tuple(int(s) for s in shape)
    if len(shape) == 0:
        raise ValueError("a 0-d parameter cannot be sharded on dim 0")
    return shape[0], math.prod(shape[1:]) if len(shape) > 1 else 1


def _stream_handle(stream, *groups) -> int:
    """The HIP stream handle of ``stream`` (torch's current stream when None),
    after checking that every non-empty tensor in ``groups`` lives on one
    device, the stream's when the stream is a torch stream: the kernels
    dereference every pointer on the device they run on."""
    if stream is None:
        stream = torch.cuda.current_stream()
    if hasattr(stream, "cuda_stream"):
        handle, device = int(stream.cuda_stream), stream.device
    else:
        handle, device = int(stream), None
    _check_device(device, groups)
    return handle


def _check_device(device, groups) -> None:
    seen = device
    for group in groups:
        for t in group:
            if t is None or t.numel() == 0:
                continue
            if seen is None:
                seen = t.device
            elif t.device != seen:
                raise ValueError(f"a tensor on {t.device} where {seen} is expected: "
                                 "one call's tensors and stream must share one device")


def _ptr_array(tensors, expect_elems, dtypes, what) -> ctypes.Array:
    arr = (ctypes.c_void_p * len(tensors))()
    for p, t in enumerate(tensors):
        if t is None:
            if expect_elems[p] != 0:
                raise ValueError(f"{what}[{p}] is None but needs {expect_elems[p]} elements")
            arr[p] = None
            continue
        if not isinstance(t, torch.Tensor) or t.dtype not in dtypes:
            raise TypeError(f"{what}[{p}] must be a tensor of dtype {dtypes}")
        if t.numel() != expect_elems[p]:
            raise ValueError(f"{what}[{p}] has {t.numel()} elements, expected {expect_elems[p]}")
        if t.numel() and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError(f"{what}[{p}] must be a contiguous device tensor")
        arr[p] = t.data_ptr() if t.numel() else None
    return arr


def _bucket_ptr(t: torch.Tensor, elems: int, dtypes, what) -> int:
    if not isinstance(t, torch.Tensor) or t.dtype not in dtypes:
        raise TypeError(f"{what} must be a tensor of dtype {dtypes}")
    if t.numel() != elems:
        raise ValueError(f"{what} has {t.numel()} elements, expected {elems}")
    if elems and (not t.is_cuda or not t.is_contiguous()):
        raise ValueError(f"{what} must be a contiguous device tensor")
    return t.data_ptr() if elems else 0


class BucketPlan:
    """A bucket of parameters sharded on dim 0 over ``world_size`` ranks.

    ``shapes`` are the full parameter shapes (dim 0 is sharded, the trailing
    dims are flattened into ``inner``), in bucket order.  ``max_workgroups``
    (> 0) caps every launch's grid and ``reduce_tiles`` ("auto", "full" or
    "half") fixes the reduction's tile size; neither changes a result.
    """

    def __init__(self, world_size: int, shapes: Sequence, align: int = 8, max_workgroups: int = 0,
                 reduce_tiles: str = "auto"):
        self._lib = _native.load()
        dims = [_rows_inner(s) for s in shapes]
        n = len(dims)
        rows = (ctypes.c_int64 * max(n, 1))(*[d[0] for d in dims])
        inner = (ctypes.c_int64 * max(n, 1))(*[d[1] for d in dims])
        if reduce_tiles not in _native.REDUCE_TILES:
            raise ValueError("reduce_tiles must be 'auto', 'full' or 'half'")
        opts = _native.PlanOptions(int(max_workgroups), _native.REDUCE_TILES[reduce_tiles], 0)
        h = ctypes.c_void_p()
        _check(self._lib.fsdp_bucket_plan_ex(int(world_size), n, rows, inner, int(align), ctypes.byref(opts),
                                             ctypes.byref(h)),
               "fsdp_bucket_plan_ex")
        self._h = h
        self.world_size = int(world_size)
        self.num_params = n
        self.align = int(align)
        self.dims = dims
        self.chunk_elems = int(self._lib.fsdp_plan_chunk_elems(h))
        self._param = []
        for p in range(n):
            c, o, L = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
            _check(self._lib.fsdp_plan_param(h, p, ctypes.byref(c), ctypes.byref(o), ctypes.byref(L)),
                   "fsdp_plan_param")
            self._param.append((c.value, o.value, L.value))

    # ---- plan queries
    def rows_per_rank(self, p: int) -> int:
        return self._param[p][0]

    def offset(self, p: int) -> int:
        return self._param[p][1]

    def seg_elems(self, p: int) -> int:
        return self._param[p][2]

    def local_rows(self, p: int, rank: int) -> int:
        r = int(self._lib.fsdp_plan_local_rows(self._h, p, rank))
        if r < 0:
            raise ValueError(f"bad parameter {p} or rank {rank}")
        return r

    def local_elems(self, p: int, rank: int) -> int:
        return self.local_rows(p, rank) * self.dims[p][1]

    def full_elems(self, p: int) -> int:
        return self.dims[p][0] * self.dims[p][1]

    # ---- the hot path
    def ag_pack(self, rank: int, shards: Sequence[torch.Tensor], send_chunk: torch.Tensor, stream=None) -> None:
        """fp32 Shard(0) slabs of ``rank`` -> bf16 send chunk of S elements."""
        self._check_len(shards, "shards")
        arr = _ptr_array(shards, [self.local_elems(p, rank) for p in range(self.num_params)],
                         (torch.float32,), "shards")
        dst = _bucket_ptr(send_chunk, self.chunk_elems, BF16_DTYPES, "send_chunk")
        h = _stream_handle(stream, shards, [send_chunk])
        _check(self._lib.fsdp_ag_pack(self._h, int(rank), arr, dst, h), "fsdp_ag_pack")

    def ag_unpack(self, gathered: torch.Tensor, params: Sequence[torch.Tensor], stream=None) -> None:
        """Rank-major W*S bf16 buffer -> full bf16 parameters."""
        self._check_len(params, "params")
        src = _bucket_ptr(gathered, self.world_size * self.chunk_elems, BF16_DTYPES, "gathered")
        arr = _ptr_array(params, [self.full_elems(p) for p in range(self.num_params)], BF16_DTYPES, "params")
        h = _stream_handle(stream, [gathered], params)
        _check(self._lib.fsdp_ag_unpack(self._h, src, arr, h), "fsdp_ag_unpack")

    def rs_pack(self, grads: Sequence[torch.Tensor], send_buf: torch.Tensor, stream=None) -> None:
        """Full bf16 gradients -> destination-major W*S bf16 send buffer."""
        self._check_len(grads, "grads")
        arr = _ptr_array(grads, [self.full_elems(p) for p in range(self.num_params)], BF16_DTYPES, "grads")
        dst = _bucket_ptr(send_buf, self.world_size * self.chunk_elems, BF16_DTYPES, "send_buf")
        h = _stream_handle(stream, grads, [send_buf])
        _check(self._lib.fsdp_rs_pack(self._h, arr, dst, h), "fsdp_rs_pack")

    def rs_reduce(self, rank: int, recv: torch.Tensor, grad_shards: Sequence[torch.Tensor], stream=None) -> None:
        """Source-major W*S bf16 buffer -> fp32 gradient shards of ``rank`` (average over ranks)."""
        self._check_len(grad_shards, "grad_shards")
        src = _bucket_ptr(recv, self.world_size * self.chunk_elems, BF16_DTYPES, "recv")
        arr = _ptr_array(grad_shards, [self.local_elems(p, rank) for p in range(self.num_params)],
                         (torch.float32,), "grad_shards")
        h = _stream_handle(stream, [recv], grad_shards)
        _check(self._lib.fsdp_rs_reduce(self._h, int(rank), src, arr, h), "fsdp_rs_reduce")

    # ---- element-type and chunk-table forms
    def ag_pack_ex(self, rank: int, shards: Sequence[torch.Tensor], send_chunk: torch.Tensor,
                   param_dtype: str = "bf16", stream=None) -> None:
        """fp32 shards -> a chunk of ``param_dtype`` ("bf16" or "f16" cast, or "f32" copy)."""
        self._check_len(shards, "shards")
        arr = _ptr_array(shards, [self.local_elems(p, rank) for p in range(self.num_params)],
                         (torch.float32,), "shards")
        dst = _bucket_ptr(send_chunk, self.chunk_elems, _elem_dtypes(param_dtype), "send_chunk")
        _check(self._lib.fsdp_ag_pack_ex(self._h, int(rank), arr, _dtype_code(param_dtype), dst,
                                         _stream_handle(stream, shards, [send_chunk])), "fsdp_ag_pack_ex")

    def ag_pack_push(self, rank: int, shards: Sequence[torch.Tensor], chunks: Sequence[torch.Tensor],
                     param_dtype: str = "bf16", stream=None) -> None:
        """fp32 shards -> the packed chunk of ``param_dtype``, written to each of the W
        ``chunks`` (where every rank receives this rank's chunk)."""
        self._check_len(shards, "shards")
        arr = _ptr_array(shards, [self.local_elems(p, rank) for p in range(self.num_params)],
                         (torch.float32,), "shards")
        carr = self._chunk_array(chunks, _elem_dtypes(param_dtype))
        _check(self._lib.fsdp_ag_pack_push(self._h, int(rank), arr, _dtype_code(param_dtype), carr,
                                           _stream_handle(stream, shards, chunks)), "fsdp_ag_pack_push")

    def ag_unpack_ex(self, chunks: Sequence[torch.Tensor], params: Sequence[torch.Tensor],
                     param_dtype: str = "bf16", stream=None) -> None:
        """W gathered chunks (rank i's at chunks[i]) -> full parameters of ``param_dtype``."""
        self._check_len(params, "params")
        carr = self._chunk_array(chunks, _elem_dtypes(param_dtype))
        arr = _ptr_array(params, [self.full_elems(p) for p in range(self.num_params)],
                         _elem_dtypes(param_dtype), "params")
        _check(self._lib.fsdp_ag_unpack_ex(self._h, _dtype_code(param_dtype), carr, arr,
                                           _stream_handle(stream, chunks, params)), "fsdp_ag_unpack_ex")

    def rs_pack_ex(self, grads: Sequence[torch.Tensor], chunks: Sequence[torch.Tensor],
                   reduce_dtype: str = "bf16", stream=None) -> None:
        """Full gradients (bf16, f16 or fp32) -> W destination chunks of ``reduce_dtype``
        (the gradients' type, or "f32")."""
        self._check_len(grads, "grads")
        names = {_dtype_name(g) for g in grads if g is not None}
        if len(names) > 1:
            raise TypeError("all gradients must have one dtype")
        gname = names.pop() if names else "bf16"
        arr = _ptr_array(grads, [self.full_elems(p) for p in range(self.num_params)], _elem_dtypes(gname), "grads")
        carr = self._chunk_array(chunks, _elem_dtypes(reduce_dtype))
        _check(self._lib.fsdp_rs_pack_ex(self._h, _dtype_code(gname), arr, _dtype_code(reduce_dtype), carr,
                                         _stream_handle(stream, grads, chunks)), "fsdp_rs_pack_ex")

    def rs_reduce_ex(self, rank: int, chunks: Sequence[torch.Tensor], grad_shards: Sequence[torch.Tensor],
                     reduce_dtype: str = "bf16", stream=None) -> None:
        """W received chunks (source i's at chunks[i]) of ``reduce_dtype`` -> fp32 shards of ``rank``."""
        self._check_len(grad_shards, "grad_shards")
        carr = self._chunk_array(chunks, _elem_dtypes(reduce_dtype))
        arr = _ptr_array(grad_shards, [self.local_elems(p, rank) for p in range(self.num_params)],
                         (torch.float32,), "grad_shards")
        _check(self._lib.fsdp_rs_reduce_ex(self._h, int(rank), _dtype_code(reduce_dtype), carr, arr,
                                           _stream_handle(stream, chunks, grad_shards)), "fsdp_rs_reduce_ex")

    def _chunk_array(self, chunks, dtypes) -> ctypes.Array:
        if len(chunks) != self.world_size:
            raise ValueError(f"{len(chunks)} chunks for world size {self.world_size}")
        arr = (ctypes.c_void_p * len(chunks))()
        for i, c in enumerate(chunks):
            arr[i] = _bucket_ptr(c, self.chunk_elems, dtypes, f"chunks[{i}]") or None
        return arr

    # ---- housekeeping
    def _check_len(self, seq, what):
        if len(seq) != self.num_params:
            raise ValueError(f"{what} has {len(seq)} entries, the plan has {self.num_params} parameters")

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.fsdp_plan_free(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
