"""Property tests of the oracle: the per-element brute-force pins of
``oracle_checks`` over random small buckets.

The strategy spans the world sizes 1, 2, 3, 4, 7, 8, 48 and 64, row counts at
the edges of the Shard(0) split (0, 1, W-1, W, W+1 and random), inner sizes
1, 3, 8 and 64, and the alignments 1 (dense) and 8.  Sizes stay small because
the checks loop over elements in Python.
"""

from __future__ import annotations

import numpy as np
from hypothesis import given, settings, strategies as st

import oracle.fsdp_oracle as O
import oracle_checks as C

WORLDS = [1, 2, 3, 4, 7, 8, 48, 64]


@st.composite
def buckets(draw):
    w = draw(st.sampled_from(WORLDS))
    nparams = draw(st.integers(1, 4))
    dims = []
    for _ in range(nparams):
        n = draw(st.sampled_from([0, 1, max(w - 1, 0), w, w + 1, draw(st.integers(0, 3 * w + 5))]))
        k = draw(st.sampled_from([1, 3, 8, 64]))
        dims.append((n, k))
    # keep the element loops of the checks short
    while sum(n * k for n, k in dims) > 6000:
        dims = [(n // 2, k) for n, k in dims]
    align = draw(st.sampled_from([1, 8]))
    rank = draw(st.integers(0, w - 1))
    seed = draw(st.integers(0, 2**16))
    return w, dims, align, rank, seed


@settings(max_examples=60, deadline=None)
@given(buckets())
def test_ag_path_by_brute_force(b):
    w, dims, align, rank, seed = b
    C.check_ag_pack_bruteforce(O, w, dims, rank, seed, align)
    C.check_ag_unpack_bruteforce(O, w, dims, seed, align)
    C.check_roundtrip_library(O, w, dims, seed, align)


@settings(max_examples=60, deadline=None)
@given(buckets())
def test_rs_path_by_brute_force(b):
    w, dims, align, rank, seed = b
    C.check_rs_pack_bruteforce(O, w, dims, seed, align)
    C.check_rs_pack_equals_ag_layout(O, w, dims, seed, align)
    C.check_rs_reduce_bruteforce(O, w, dims, rank, seed, align)


@settings(max_examples=60, deadline=None)
@given(buckets())
def test_plan_matches_torch_chunk(b):
    w, dims, align, _, _ = b
    plan = O.make_plan(w, dims, align)
    for p, (n, _) in enumerate(dims):
        assert [O.local_rows(plan, p, r) for r in range(w)] == C.torch_chunk_rows(n, w)
    # segments are aligned, disjoint, in caller order, and the chunk ends aligned
    ends = [plan.offset[p] + plan.rows_per_rank[p] * k for p, (_, k) in enumerate(dims)]
    assert all(o % align == 0 for o in plan.offset) and plan.chunk % align == 0
    assert all(ends[p] <= plan.offset[p + 1] for p in range(len(dims) - 1))
    assert ends[-1] <= plan.chunk < ends[-1] + align
    assert np.all(np.diff(plan.offset) >= 0)
