"""Seeded value generators.

Every generator draws from its own ``numpy`` PCG64 stream keyed by a tuple of
integers, so any slab of rows can be produced without producing the rest of
the tensor (a 405B-block parameter has 872M elements).  Rows are grouped in
blocks of about 2**20 elements; block ``b`` of a tensor always comes from the
same stream, whatever slab is asked for.

Values:
* parameters: N(0, 1) * 0.02 in fp32; RMSNorm weights are 1.0;
* gradients: N(0, 1) * 1e-3 drawn in fp32 and turned into bf16 bit patterns
  by keeping the upper 16 bits (truncation: a generator choice that keeps the
  distribution, not the method's round-to-nearest-even);
* raw bit patterns (uniform over all 16- or 32-bit words, NaNs and
  infinities included) for special-value coverage.
"""

from __future__ import annotations

import numpy as np

BLOCK_ELEMS = 1 << 20
PARAM_SCALE = np.float32(0.02)
GRAD_SCALE = np.float32(1e-3)


def _rng(words) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(w) for w in words])))


def _rows_per_block(inner: int) -> int:
    return max(1, BLOCK_ELEMS // max(1, inner))


def _normal_rows(prefix, lo: int, hi: int, inner: int) -> np.ndarray:
    """Rows [lo, hi) of a (rows, inner) tensor of N(0,1) fp32 values."""
    out = np.empty((max(0, hi - lo), inner), dtype=np.float32)
    if hi <= lo:
        return out
    rpb = _rows_per_block(inner)
    b0, b1 = lo // rpb, (hi - 1) // rpb
    for b in range(b0, b1 + 1):
        blk = _rng(list(prefix) + [b]).standard_normal(rpb * inner, dtype=np.float32)
        blk = blk.reshape(rpb, inner)
        r0 = max(lo, b * rpb)
        r1 = min(hi, (b + 1) * rpb)
        out[r0 - lo:r1 - lo] = blk[r0 - b * rpb:r1 - b * rpb]
    return out


def param_rows(key: int, p: int, lo: int, hi: int, inner: int, is_norm: bool = False) -> np.ndarray:
    """fp32 rows [lo, hi) of parameter ``p`` of workload ``key``."""
    if is_norm:
        return np.ones((max(0, hi - lo), inner), dtype=np.float32)
    x = _normal_rows((key, 0, p), lo, hi, inner)
    x *= PARAM_SCALE
    return x


def grad_rows_bits(key: int, src_rank: int, p: int, lo: int, hi: int, inner: int) -> np.ndarray:
    """bf16 bit patterns (uint16) of rows [lo, hi) of rank ``src_rank``'s gradient of ``p``."""
    g = _normal_rows((key, 1, src_rank, p), lo, hi, inner)
    g *= GRAD_SCALE
    return (g.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def random_bits16(words, n: int) -> np.ndarray:
    """``n`` uniformly random 16-bit words."""
    return np.frombuffer(_rng(words).bytes(2 * n), dtype=np.uint16).copy()


def random_bits32(words, n: int) -> np.ndarray:
    """``n`` uniformly random 32-bit words (reinterpret as fp32 for all-pattern inputs)."""
    return np.frombuffer(_rng(words).bytes(4 * n), dtype=np.uint32).copy()


def exact_grad_bits(words, shape) -> np.ndarray:
    """bf16 bit patterns of k/64 with integer k in [-200, 200].

    Such values are exact in bf16, and any sum of up to 2**16 of them is exact
    in fp32, so a reduction of them has one correct answer in any order.
    """
    k = _rng(words).integers(-200, 201, size=shape)
    f = (k.astype(np.float32) / np.float32(64.0)).astype(np.float32)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
