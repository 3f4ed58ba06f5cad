"""CPU oracle for one rank's share of SimpleFSDP's bucketed communication path.

TEST INFRASTRUCTURE ONLY.  This module is the plain, slow, obviously correct
definition that the GPU kernels are checked against.  Only the test suite,
the smoke check and the benchmark's CPU-baseline leg may import it; the
product path (the C-ABI library and its Python binding) never does, and it
shares no code with that path.

What is computed (SimpleFSDP, arXiv 2411.00284):

* Sharding (section 3.1; section 2.1 "Model Initialization & Parameter
  Sharding"): every parameter is a DTensor placed ``Shard(0)`` over the
  data-parallel ranks.  A dim-0 of N rows over W ranks is split like
  ``torch.chunk``: c = ceil(N / W) rows per rank, rank r holding
  n_r = min(c, max(0, N - r*c)) rows (the last ranks may hold fewer or none).
* All-gather with mixed precision (section 4, "Mixed precision training" and
  its ``replicate_compute`` listing): ``Shard(0) -> Replicate`` with
  ``forward_dtype = param_dtype``, a 16-bit float.  The result on every rank is
  the full parameter cast to bf16.
* Reduce-scatter (same listing, ``grad_placements = Partial("avg")``): rank j
  receives dim-0 chunk j of the average over ranks of the per-rank gradients,
  reduced in ``reduce_dtype`` = fp32.
* Bucketing (section 3.2.1): the all-gather inputs of a bucket are flattened
  and concatenated into one larger buffer (copy-in), gathered, and copied out
  by each parameter's original size; for the reduce-scatter every gradient is
  split into W chunks and the chunks are concatenated per destination rank,
  the bucket is reduce-scattered with averaging, and each rank reads its
  gradients out of the reduced buffer.

Readings where the paper is silent:

* bucket layout: parameters in caller order; parameter p starts at off_p,
  a multiple of the alignment ``align`` (elements); each per-rank chunk has
  S elements; pad rows, alignment gaps and the chunk tail hold +0.0;
* the 16-bit format is bf16 with IEEE-754 round-half-to-even; a NaN maps to
  a quiet NaN of the same sign (payload not part of the contract); fp16
  (IEEE binary16, also round-half-to-even, with subnormals and overflow to
  infinity) is the other 16-bit float the paper's wording allows, and is
  supported as a param_dtype / reduce_dtype too;
* the gathered buffer is rank-major [W][S]; the reduce-scatter send buffer is
  destination-major [W][S];
* the average: fp32 sum over source ranks 0..W-1 in that order, starting
  from the rank-0 value, then one correctly rounded division by W;
* all fp32 arithmetic keeps subnormals (numpy does not flush them).

Representation: bf16 data is held as ``uint16`` bit patterns, fp16 data as
``numpy.float16``, fp32 data as ``numpy.float32``.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Sequence

import numpy as np

__all__ = [
    "Plan",
    "make_plan",
    "local_rows",
    "local_elems",
    "bf16_rne",
    "bf16_to_f32",
    "f16_rne",
    "ag_pack",
    "all_gather",
    "ag_unpack",
    "rs_pack",
    "rs_exchange",
    "rs_reduce",
    "ag_pack_range",
    "ag_unpack_rows",
    "rs_pack_range",
    "rs_reduce_range",
]


# --------------------------------------------------------------------------
# O0: the bucket plan
# --------------------------------------------------------------------------

def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def _round_up(a: int, m: int) -> int:
    return _ceil_div(a, m) * m


@dataclass(frozen=True)
class Plan:
    """Layout of one bucket for world size W (all sizes in elements).

    rows[p], inner[p]   parameter p has shape (rows, inner), row-major
    rows_per_rank[p]    c_p = ceil(rows / W): dim-0 rows of one Shard(0) chunk
    seg[p]              L_p = c_p * inner: elements of p in every rank's chunk
    offset[p]           off_p: where p starts inside a rank's chunk
    chunk               S: elements of one rank's chunk (a multiple of align)
    """

    world_size: int
    align: int
    rows: tuple[int, ...]
    inner: tuple[int, ...]
    rows_per_rank: tuple[int, ...]
    seg: tuple[int, ...]
    offset: tuple[int, ...]
    chunk: int

    @property
    def num_params(self) -> int:
        return len(self.rows)


def make_plan(world_size: int, dims: Sequence[tuple[int, int]], align: int = 8) -> Plan:
    """Plan a bucket: parameters concatenated in the given order (section 3.2.1).

    Each parameter is padded along dim 0 to W * c_p rows, so that every rank's
    chunk holds the same L_p elements of it; each parameter starts at the next
    multiple of ``align``, and S is the end of the last parameter rounded up to
    ``align``.  ``align = 1`` gives the dense flatten-and-concatenate buffer.
    """
    if world_size < 1:
        raise ValueError("world_size must be >= 1")
    if align < 1 or (align & (align - 1)):
        raise ValueError("align must be a power of two")
    if len(dims) < 1:
        raise ValueError("a bucket needs at least one parameter")
    rows, inner, cpr, seg, off = [], [], [], [], []
    pos = 0
    for n, k in dims:
        n, k = int(n), int(k)
        if n < 0 or k < 1:
            raise ValueError("rows must be >= 0 and inner >= 1")
        c = _ceil_div(n, world_size)
        pos = _round_up(pos, align)
        rows.append(n)
        inner.append(k)
        cpr.append(c)
        seg.append(c * k)
        off.append(pos)
        pos += c * k
    chunk = _round_up(pos, align)
    return Plan(world_size, align, tuple(rows), tuple(inner), tuple(cpr),
                tuple(seg), tuple(off), chunk)


def local_rows(plan: Plan, p: int, rank: int) -> int:
    """n_{p,rank}: rows of parameter p held by ``rank`` (torch.chunk split)."""
    c = plan.rows_per_rank[p]
    return min(c, max(0, plan.rows[p] - rank * c))


def local_elems(plan: Plan, p: int, rank: int) -> int:
    return local_rows(plan, p, rank) * plan.inner[p]


# --------------------------------------------------------------------------
# bf16 encoding
# --------------------------------------------------------------------------

def bf16_rne(x) -> np.ndarray:
    """fp32 -> bf16 bit patterns, IEEE-754 round-half-to-even.

    bf16 keeps the upper 16 bits of the fp32 word.  The 16 dropped bits are
    rounded to nearest with ties to an even kept mantissa: adding 0x7FFF plus
    the lowest kept bit and truncating carries into the kept part exactly when
    the dropped part is above half, or equal to half with an odd kept part.
    A carry out of the mantissa moves to the next binade and, from the largest
    finite values, to infinity; subnormals and zeros follow the same rule.
    NaN inputs give a quiet NaN with the input's sign.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) & np.uint64(0xFFFF)
    is_nan = (u & np.uint64(0x7FFFFFFF)) > np.uint64(0x7F800000)
    qnan = ((u >> np.uint64(16)) | np.uint64(0x0040)) & np.uint64(0xFFFF)
    r = np.where(is_nan, qnan, r)
    return r.astype(np.uint16).reshape(np.shape(x))


def bf16_to_f32(bits) -> np.ndarray:
    """bf16 bit patterns -> fp32 values (exact: the low 16 bits are zero)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f16_rne(x) -> np.ndarray:
    """fp32 -> IEEE-754 binary16 (fp16) values, round-half-to-even.

    numpy's float32 -> float16 conversion, a library routine: the nearest
    binary16 value with ties to an even significand, subnormals below 2^-14,
    +-0 below half the smallest subnormal, and infinity from 65520 (the
    largest finite value plus half an ulp) up.  A NaN gives a NaN; its payload
    is not part of the contract.
    """
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float32).astype(np.float16)


# --------------------------------------------------------------------------
# Forward: all-gather copy-in / exchange / copy-out
# --------------------------------------------------------------------------

def ag_pack(plan: Plan, rank: int, shards: Sequence[np.ndarray], param_dtype: str = "bf16") -> np.ndarray:
    """O1, all-gather copy-in of one rank (section 3.2.1; section 4 param_dtype).

    ``shards[p]`` is the rank's unpadded fp32 Shard(0) slab of parameter p,
    n_{p,rank} x inner_p.  Output: the rank's chunk of S elements, with shard p
    cast to ``param_dtype`` at off_p and zeros everywhere else (pad rows, gaps,
    tail).  ``param_dtype`` is "bf16" (mixed precision: bf16 bit patterns as
    uint16), "f16" (mixed precision with fp16: numpy float16 values) or "f32"
    (no mixed precision: the fp32 values themselves).
    """
    if not 0 <= rank < plan.world_size:
        raise ValueError("rank out of range")
    out_dtype = _wire_dtype(param_dtype)
    send = np.zeros(plan.chunk, dtype=out_dtype)
    for p in range(plan.num_params):
        v = local_elems(plan, p, rank)
        src = np.asarray(shards[p], dtype=np.float32).reshape(-1)
        if src.size != v:
            raise ValueError(f"shard {p} has {src.size} elements, expected {v}")
        o = plan.offset[p]
        if param_dtype == "bf16":
            send[o:o + v] = bf16_rne(src)
        elif param_dtype == "f16":
            send[o:o + v] = f16_rne(src)
        else:
            send[o:o + v] = src
    return send


def _wire_dtype(name: str):
    if name == "bf16":
        return np.uint16
    if name == "f16":
        return np.float16
    if name == "f32":
        return np.float32
    raise ValueError("dtype must be 'bf16', 'f16' or 'f32'")


def all_gather(chunks: Sequence[np.ndarray]) -> np.ndarray:
    """O2, the exchange (not on the GPU path): gathered[i*S + k] = chunk_i[k]."""
    return np.concatenate([np.asarray(c).reshape(-1) for c in chunks])


def ag_unpack(plan: Plan, gathered: np.ndarray) -> list[np.ndarray]:
    """O3, all-gather copy-out ("copy out ... based on their original tensor size").

    Row ``row`` of parameter p came from rank i = row // c_p, where it sat at
    row q = row % c_p of p's segment: element (row, col) is
    gathered[i*S + off_p + q*inner_p + col].  Rows of one rank are contiguous
    on both sides, so each rank's rows move as one slice.  Output: the full,
    unpadded parameters, rows x inner, in the gathered buffer's element type
    (bf16 bit patterns or fp32).
    """
    W, S = plan.world_size, plan.chunk
    g = np.asarray(gathered).reshape(-1)
    if g.size != W * S:
        raise ValueError("gathered buffer must hold W*S elements")
    out = []
    for p in range(plan.num_params):
        n, k, c, o = plan.rows[p], plan.inner[p], plan.rows_per_rank[p], plan.offset[p]
        full = np.empty((n, k), dtype=g.dtype)
        for i in range(W):
            ni = local_rows(plan, p, i)
            if ni == 0:
                continue
            base = i * S + o
            full[i * c:i * c + ni, :] = g[base:base + ni * k].reshape(ni, k)
        out.append(full)
    return out


# --------------------------------------------------------------------------
# Backward: reduce-scatter copy-in / exchange / reduction with read-out
# --------------------------------------------------------------------------

def rs_pack(plan: Plan, grads: Sequence[np.ndarray], reduce_dtype: str | None = None) -> np.ndarray:
    """O4, reduce-scatter copy-in (section 3.2.1; section 4 reduce_dtype).

    Each full gradient G_p (rows x inner) is zero-padded along dim 0 to
    W * c_p rows and split into W chunks of c_p rows; chunk j goes to
    destination j's part of the send buffer at j*S + off_p.  Everything the
    chunks do not cover is zero.  Gradients are bf16 bit patterns (uint16),
    fp16 or fp32.  ``reduce_dtype="f32"`` casts 16-bit gradients to fp32 first
    (an exact widening); by default the buffer keeps the gradients' own type.
    """
    W, S = plan.world_size, plan.chunk
    gs = [np.asarray(g) for g in grads]
    if reduce_dtype == "f32":
        gs = [bf16_to_f32(g) if g.dtype == np.uint16 else g.astype(np.float32) for g in gs]
    elif reduce_dtype not in (None, "bf16", "f16"):
        raise ValueError("reduce_dtype must be 'bf16', 'f16' or 'f32'")
    dtype = gs[0].dtype if gs else np.uint16
    if reduce_dtype == "bf16" and dtype != np.uint16:
        raise ValueError("a bf16 wire needs bf16 gradients")
    if reduce_dtype == "f16" and dtype != np.float16:
        raise ValueError("an fp16 wire needs fp16 gradients")
    send = np.zeros(W * S, dtype=dtype)
    for p in range(plan.num_params):
        n, k, c, L, o = (plan.rows[p], plan.inner[p], plan.rows_per_rank[p],
                         plan.seg[p], plan.offset[p])
        G = gs[p].astype(dtype, copy=False).reshape(n, k)
        padded = np.zeros((W * c, k), dtype=dtype)
        padded[:n] = G
        flat = padded.reshape(-1)
        for j in range(W):
            send[j * S + o:j * S + o + L] = flat[j * L:(j + 1) * L]
    return send


def rs_exchange(send_bufs: Sequence[np.ndarray], rank: int, chunk: int) -> np.ndarray:
    """O5, the exchange (not on the GPU path): recv[i*S + k] = send_i[rank*S + k]."""
    return np.concatenate([np.asarray(b).reshape(-1)[rank * chunk:(rank + 1) * chunk]
                           for b in send_bufs])


def rs_reduce(plan: Plan, rank: int, recv: np.ndarray) -> list[np.ndarray]:
    """O6, the rank-local average and read-out (section 3.2.1; section 4 reduce_dtype).

    For every element of the rank's Shard(0) slab of parameter p: take the W
    incoming values x_0..x_{W-1} in fp32 (bf16 bit patterns and fp16 values
    are widened, exactly; an fp32 buffer is used as it is), start from x_0, add x_1, ...,
    x_{W-1} one at a time in fp32, then divide once by W in fp32.  Output: the
    fp32 gradient shards, n_{p,rank} x inner_p (no padded rows).
    """
    W, S = plan.world_size, plan.chunk
    if not 0 <= rank < W:
        raise ValueError("rank out of range")
    r = np.asarray(recv).reshape(-1)
    widen = bf16_to_f32 if r.dtype == np.uint16 else (lambda a: np.asarray(a, dtype=np.float32))
    if r.size != W * S:
        raise ValueError("recv buffer must hold W*S elements")
    wf = np.float32(W)
    out = []
    for p in range(plan.num_params):
        n, k, o = local_rows(plan, p, rank), plan.inner[p], plan.offset[p]
        v = n * k
        acc = widen(r[o:o + v]).copy()
        for i in range(1, W):
            x = widen(r[i * S + o:i * S + o + v])
            acc = np.add(acc, x, dtype=np.float32)
        res = np.divide(acc, wf, dtype=np.float32)
        out.append(res.reshape(n, k))
    return out


# --------------------------------------------------------------------------
# The same definitions for a slice of one output, reading only the inputs
# that slice depends on (for buckets too large to hold several copies of on
# the host).  ``read(...)`` callbacks return input elements as numpy arrays.
# --------------------------------------------------------------------------

def ag_pack_range(plan: Plan, rank: int, read_shard, k0: int, k1: int) -> np.ndarray:
    """O1 restricted to send[k0:k1]; read_shard(p, lo, hi) -> fp32 shard p[lo:hi]."""
    out = np.zeros(max(0, k1 - k0), dtype=np.uint16)
    for p in range(plan.num_params):
        o, v = plan.offset[p], local_elems(plan, p, rank)
        lo, hi = max(k0, o), min(k1, o + v)
        if lo < hi:
            out[lo - k0:hi - k0] = bf16_rne(read_shard(p, lo - o, hi - o))
    return out


def ag_unpack_rows(plan: Plan, read_gathered, p: int, rows) -> np.ndarray:
    """O3 for the listed rows of parameter p; read_gathered(start, count) ->
    gathered[start:start+count]."""
    k, c, o, S = plan.inner[p], plan.rows_per_rank[p], plan.offset[p], plan.chunk
    out = np.empty((len(rows), k), dtype=np.uint16)
    for t, row in enumerate(rows):
        if not 0 <= row < plan.rows[p]:
            raise ValueError("row out of range")
        i, q = divmod(int(row), c)
        out[t] = read_gathered(i * S + o + q * k, k)
    return out


def rs_pack_range(plan: Plan, read_grad, j: int, k0: int, k1: int) -> np.ndarray:
    """O4 restricted to send[j*S + k0 : j*S + k1]; read_grad(p, lo, hi) ->
    flattened bf16 gradient p[lo:hi]."""
    out = np.zeros(max(0, k1 - k0), dtype=np.uint16)
    for p in range(plan.num_params):
        o, L, k = plan.offset[p], plan.seg[p], plan.inner[p]
        valid = local_rows(plan, p, j) * k          # rows j*c .. that exist
        lo, hi = max(k0, o), min(k1, o + min(L, valid))
        if lo < hi:
            out[lo - k0:hi - k0] = read_grad(p, j * L + (lo - o), j * L + (hi - o))
    return out


def rs_reduce_range(plan: Plan, rank: int, read_recv, p: int, e0: int, e1: int) -> np.ndarray:
    """O6 for elements [e0, e1) of parameter p's output shard; read_recv(start,
    count) -> recv[start:start+count]."""
    W, S, o = plan.world_size, plan.chunk, plan.offset[p]
    if not 0 <= e0 <= e1 <= local_elems(plan, p, rank):
        raise ValueError("range outside the shard")
    acc = bf16_to_f32(read_recv(o + e0, e1 - e0))
    for i in range(1, W):
        acc = np.add(acc, bf16_to_f32(read_recv(i * S + o + e0, e1 - e0)), dtype=np.float32)
    return np.divide(acc, np.float32(W), dtype=np.float32)
