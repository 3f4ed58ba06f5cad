"""Parameter shapes of the synthetic workloads (one transformer block per bucket).

Each parameter is described by ``(rows, inner)``: ``rows`` is dim 0 (the
dimension FSDP shards, paper section 3.1) and ``inner`` is the product of all
trailing dimensions (1 for a 1-D tensor such as an RMSNorm weight).
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

BLOCK_NAMES = ("wq", "wk", "wv", "wo", "w1", "w2", "w3", "attention_norm", "ffn_norm")
KV_ROWS = 1024          # 8 key/value heads x head dim 128 (Llama 3.1, all sizes)
VOCAB = 128256          # Llama 3 vocabulary


@dataclass(frozen=True)
class Workload:
    """One bucket: a simulated world size and the parameters it concatenates."""

    key: int
    name: str
    world_size: int
    names: tuple[str, ...]
    dims: tuple[tuple[int, int], ...]     # (rows, inner) per parameter
    is_norm: tuple[bool, ...]             # RMSNorm weights are initialised to 1.0

    @property
    def num_params(self) -> int:
        return len(self.dims)

    @property
    def total_elems(self) -> int:
        return sum(n * k for n, k in self.dims)


def _block(key: int, name: str, world_size: int, dim: int, ffn: int, kv_rows: int) -> Workload:
    dims = (
        (dim, dim),        # wq
        (kv_rows, dim),    # wk
        (kv_rows, dim),    # wv
        (dim, dim),        # wo
        (ffn, dim),        # w1
        (dim, ffn),        # w2
        (ffn, dim),        # w3
        (dim, 1),          # attention_norm
        (dim, 1),          # ffn_norm
    )
    return Workload(key, name, world_size, BLOCK_NAMES, dims,
                    tuple(n.endswith("norm") for n in BLOCK_NAMES))


def _block_tp(key: int, name: str, world_size: int, dim: int, ffn: int, kv_rows: int, tp: int) -> Workload:
    """One block's tensor-parallel shards as an FSDP bucket on the data-parallel
    sub-mesh (paper section 4, tensor parallel: each parameter is a 2-D DTensor
    and the all-gather runs over the DP sub-mesh only; section 5 trains the 70B
    model with TP degree 8).  The Megatron split: wq, wk, wv, w1 and w3 are
    column-parallel (their output rows split over the TP group), wo and w2
    row-parallel (their input columns split), the norm weights replicated."""
    dims = (
        (dim // tp, dim),        # wq
        (kv_rows // tp, dim),    # wk
        (kv_rows // tp, dim),    # wv
        (dim, dim // tp),        # wo
        (ffn // tp, dim),        # w1
        (dim, ffn // tp),        # w2
        (ffn // tp, dim),        # w3
        (dim, 1),                # attention_norm
        (dim, 1),                # ffn_norm
    )
    return Workload(key, name, world_size, BLOCK_NAMES, dims,
                    tuple(n.endswith("norm") for n in BLOCK_NAMES))


def _uneven(key: int) -> Workload:
    """Embedding, output projection, final norm and 37 odd-sized tensors.

    The odd shapes are drawn once from a fixed numpy stream: dim 0 uniform in
    [1, 5000] and dim 1 chosen from {1, 4096}.
    """
    rng = np.random.default_rng(np.random.SeedSequence([key, 0]))
    d0 = rng.integers(1, 5001, 37)
    d1 = rng.choice([1, 4096], 37)
    names = ["tok_embeddings", "output", "norm"] + [f"odd_{i}" for i in range(37)]
    dims = [(VOCAB, 4096), (VOCAB, 4096), (4096, 1)]
    dims += [(int(a), int(b)) for a, b in zip(d0, d1)]
    is_norm = [False, False, True] + [False] * 37
    return Workload(key, "uneven-embed-odd40-w48", 48, tuple(names), tuple(dims), tuple(is_norm))


WORKLOADS: dict[int, Workload] = {
    1: _block(1, "toy-block-w4", 4, dim=256, ffn=688, kv_rows=256),
    2: _block(2, "llama3-8b-block-w8", 8, dim=4096, ffn=14336, kv_rows=KV_ROWS),
    3: _block(3, "llama3-70b-block-w64", 64, dim=8192, ffn=28672, kv_rows=KV_ROWS),
    4: _block(4, "llama3-405b-block-w128", 128, dim=16384, ffn=53248, kv_rows=KV_ROWS),
    5: _uneven(5),
    # 64 GPUs as TP 8 x DP 8: the bucket holds one TP rank's shards, W = 8
    6: _block_tp(6, "llama3-70b-block-tp8-w8", 8, dim=8192, ffn=28672, kv_rows=KV_ROWS, tp=8),
    # the 8B block under FSDP alone on 128 GPUs (the largest FSDP-only setting of section 5)
    7: _block(7, "llama3-8b-block-w128", 128, dim=4096, ffn=14336, kv_rows=KV_ROWS),
}


def workload(key: int) -> Workload:
    return WORKLOADS[key]
