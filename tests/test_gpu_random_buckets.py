"""GPU parity on seeded random buckets: world sizes 1-128, 1-64 parameters
of random shapes (empty, 1-wide, dim 0 below W, several tiles), every
alignment 1-16, element-aligned parameter pointers, random ranks.  Every
kernel and every element-type, chunk-table and push form is compared with the
oracle bit for bit, inside poisoned guard bands."""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle.fsdp_oracle as O
from gpu_util import Guarded, host_u16, host_u32, step, to_dev_f32, to_dev_u16
from synth import random_bits16, random_bits32
from test_gpu_parity import run_ag_pack, run_ag_unpack, run_rs_pack, run_rs_reduce, wide_bf16_host

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU"),
              pytest.mark.filterwarnings("ignore::RuntimeWarning")]   # NaN/inf in the oracle's sums

if torch.cuda.is_available():
    from paper_2411_00284_amd import BucketPlan

import os

# 200 by default; a longer sweep can ask for more (cases are seeded by index)
N_CASES = int(os.environ.get("FSDP_TEST_RANDOM_CASES", "200"))


def random_case(i):
    rng = np.random.default_rng([2024, i])
    W = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 13, 16, 31, 48, 64, 100, 128]))
    P = int(rng.integers(1, 65)) if rng.random() < 0.3 else int(rng.integers(1, 10))
    dims = []
    for _ in range(P):
        kind = rng.random()
        if kind < 0.1:
            n = 0
        elif kind < 0.3:
            n = int(rng.integers(1, W + 2))
        elif kind < 0.9:
            n = int(rng.integers(1, 4 * W + 40))
        else:
            n = int(rng.integers(W, 40 * W + 5000))
        k = int(rng.choice([1, 1, 2, 3, 7, 8, 64, 129, 4096]))
        if n * k > 400000:
            k = 1
        dims.append((n, k))
    align = int(rng.choice([1, 2, 4, 8, 8, 16]))
    shift = int(rng.integers(0, 2))
    ranks = sorted({int(x) for x in rng.integers(0, W, 2)})
    return W, dims, align, shift, ranks


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_bucket(i):
    W, dims, align, shift, ranks = random_case(i)
    plan = BucketPlan(W, dims, align)
    oplan = O.make_plan(W, dims, align)
    assert plan.chunk_elems == oplan.chunk
    S = oplan.chunk
    P = len(dims)
    step(f"random bucket {i}: W={W} P={P} align={align} shift={shift} ranks={ranks}")
    for r in ranks:
        run_ag_pack(plan, oplan, r, seed=1000 + i, shift=shift)
    run_ag_unpack(plan, oplan, seed=1000 + i, shift=shift)
    run_rs_pack(plan, oplan, seed=1000 + i, shift=shift)
    recv = wide_bf16_host([1000, i], W * S)
    for r in ranks:
        run_rs_reduce(plan, oplan, r, recv, shift=shift)
    # element-type and chunk-table forms at one rank
    r = ranks[-1]
    shards = [random_bits32([2000, i, p], O.local_elems(oplan, p, r)).view(np.float32) for p in range(P)]
    bufs = [Guarded(s.size, torch.float32, shift) for s in shards]
    for b, s_ in zip(bufs, shards):
        if s_.size:
            b.view.copy_(to_dev_f32(s_))
    out = Guarded(S, torch.float32)
    step(f"random bucket {i}: ag_pack_ex f32")
    plan.ag_pack_ex(r, [b.view for b in bufs], out.view, "f32")
    torch.cuda.synchronize()
    assert out.guards_intact()
    assert np.array_equal(host_u32(out.view), O.ag_pack(oplan, r, shards, "f32").view(np.uint32))
    grads = [random_bits16([3000, i, p], n * k) for p, (n, k) in enumerate(dims)]
    gbufs = [Guarded(g.size, torch.bfloat16, shift) for g in grads]
    for b, g in zip(gbufs, grads):
        if g.size:
            b.view.copy_(to_dev_u16(g))
    chunks = [Guarded(S, torch.float32) for _ in range(W)]
    step(f"random bucket {i}: rs_pack_ex bf16->f32 into {W} chunks")
    plan.rs_pack_ex([b.view for b in gbufs], [c.view for c in chunks], "f32")
    torch.cuda.synchronize()
    want = O.rs_pack(oplan, [g.reshape(n, k) for g, (n, k) in zip(grads, dims)], "f32")
    for j, c in enumerate(chunks):
        assert c.guards_intact(), j
        assert np.array_equal(host_u32(c.view), want[j * S:(j + 1) * S].view(np.uint32)), j
    # the fp32 reduce of those raw bit patterns: a NaN stays a NaN (its payload after an add is
    # not part of the contract), every other output is bit-exact
    outs = [Guarded(O.local_elems(oplan, p, r), torch.float32, shift) for p in range(P)]
    step(f"random bucket {i}: rs_reduce_ex f32 of raw bit patterns")
    plan.rs_reduce_ex(r, [c.view for c in chunks], [o.view for o in outs], "f32")
    torch.cuda.synchronize()
    wantr = O.rs_reduce(oplan, r, want)
    for p, o in enumerate(outs):
        assert o.guards_intact(), p
        got = host_u32(o.view).view(np.float32)
        ref = wantr[p].reshape(-1)
        nan = np.isnan(ref)
        assert np.array_equal(np.isnan(got), nan), p
        assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32)), p
    # the fp32 reduce on finite values
    rng = np.random.default_rng([5000, i])
    recv32 = (rng.standard_normal(W * S) * np.exp2(rng.integers(-30, 31, W * S))).astype(np.float32)
    for j, c in enumerate(chunks):
        if S:
            c.view.copy_(to_dev_f32(recv32[j * S:(j + 1) * S]))
    outs = [Guarded(O.local_elems(oplan, p, r), torch.float32, shift) for p in range(P)]
    step(f"random bucket {i}: rs_reduce_ex f32 from {W} chunks")
    plan.rs_reduce_ex(r, [c.view for c in chunks], [o.view for o in outs], "f32")
    torch.cuda.synchronize()
    wantr = O.rs_reduce(oplan, r, recv32)
    for p, o in enumerate(outs):
        assert o.guards_intact(), p
        assert np.array_equal(host_u32(o.view), wantr[p].reshape(-1).view(np.uint32)), p
    # fp16: the pack of rank r, and the reduce of finite fp16 chunks
    out16 = Guarded(S, torch.float16)
    step(f"random bucket {i}: ag_pack_ex f16")
    plan.ag_pack_ex(r, [b.view for b in bufs], out16.view, "f16")
    torch.cuda.synchronize()
    assert out16.guards_intact()
    got16 = host_u16(out16.view).view(np.float16)
    want16 = O.ag_pack(oplan, r, shards, "f16")
    nan16 = np.isnan(want16)
    assert np.array_equal(np.isnan(got16), nan16)
    assert np.array_equal(got16.view(np.uint16)[~nan16], want16.view(np.uint16)[~nan16])
    rng16 = np.random.default_rng([6000, i])
    recv16 = (rng16.integers(0, 0x7C00, W * S) | (rng16.integers(0, 2, W * S) << 15)).astype(np.uint16)
    chunks16 = [Guarded(S, torch.float16) for _ in range(W)]
    for j, c in enumerate(chunks16):
        if S:
            c.view.copy_(to_dev_u16(recv16[j * S:(j + 1) * S]).view(torch.float16))
    outs = [Guarded(O.local_elems(oplan, p, r), torch.float32, shift) for p in range(P)]
    step(f"random bucket {i}: rs_reduce_ex f16 from {W} chunks")
    plan.rs_reduce_ex(r, [c.view for c in chunks16], [o.view for o in outs], "f16")
    torch.cuda.synchronize()
    wantr = O.rs_reduce(oplan, r, recv16.view(np.float16))
    for p, o in enumerate(outs):
        assert o.guards_intact(), p
        assert np.array_equal(host_u32(o.view), wantr[p].reshape(-1).view(np.uint32)), p
    src_chunks = [Guarded(S, torch.bfloat16) for _ in range(W)]
    g = random_bits16([4000, i], W * S)
    for j, c in enumerate(src_chunks):
        if S:
            c.view.copy_(to_dev_u16(g[j * S:(j + 1) * S]))
    params = [Guarded(n * k, torch.bfloat16, shift) for n, k in dims]
    step(f"random bucket {i}: ag_unpack_ex from {W} chunks")
    plan.ag_unpack_ex([c.view for c in src_chunks], [q.view for q in params])
    torch.cuda.synchronize()
    wantu = O.ag_unpack(oplan, g)
    for p, q in enumerate(params):
        assert q.guards_intact(), p
        assert np.array_equal(host_u16(q.view), wantu[p].reshape(-1)), p
    # the bf16 pack of rank r pushed to W separate destinations (at W >= 8 a
    # pack into chunk r followed by a copy to the others)
    dsts = [Guarded(S, torch.bfloat16) for _ in range(W)]
    step(f"random bucket {i}: ag_pack_push bf16 to {W} chunks, rank {r}")
    plan.ag_pack_push(r, [b.view for b in bufs], [d.view for d in dsts])
    torch.cuda.synchronize()
    wantp = O.ag_pack(oplan, r, shards)
    for j, d in enumerate(dsts):
        assert d.guards_intact(), j
        assert np.array_equal(host_u16(d.view), wantp), j
    plan.close()
