"""GPU parity of the element-type and chunk-table entry points (the *_ex calls).

* fp32 param_dtype (training without mixed precision): ag_pack_ex copies the
  fp32 shards bit for bit, ag_unpack_ex copies fp32 chunks out.
* fp32 reduce_dtype: rs_pack_ex casts bf16 gradients to fp32 (exactly) or
  copies fp32 gradients; rs_reduce_ex sums fp32 chunks.
* chunk tables: every bucket buffer is W separate allocations (each inside
  its own poisoned guard bands), as when the chunks live on the peers.

Every output is compared with the oracle bit for bit; the chunk-table forms
with bf16 data must also agree with the contiguous calls.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle.fsdp_oracle as O
from gpu_util import (DEV, Guarded, dev_random_bits16, dev_wide_bf16, dev_wide_f32, host_u16, host_u32, step,
                      to_dev_f32, to_dev_u16)
from synth import WORKLOADS, random_bits16, random_bits32

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

if torch.cuda.is_available():
    from paper_2411_00284_amd import BucketPlan

CASES = [
    (1, [(5, 3), (1, 1), (0, 4)]),
    (3, [(7, 3), (2, 5), (10, 1), (3, 8)]),
    (4, [(16, 8), (9, 3), (3, 1), (4, 16), (1, 7)]),
    (8, [(17, 8), (8, 8), (64, 1), (1, 1)]),
    (48, [(86, 1), (4096, 1), (1, 3), (47, 2), (49, 1)]),
    (3, [(5000, 7), (4096, 4), (1, 1), (20000, 1), (2049, 8)]),
    (128, [(300, 5), (129, 8), (2, 1)]),            # the chunk-table limit
]

TORCH = {"bf16": torch.bfloat16, "f16": torch.float16, "f32": torch.float32}


def _host(t, dtype):
    if dtype == "bf16":
        return host_u16(t)
    if dtype == "f16":
        return host_u16(t).view(np.float16)
    return host_u32(t).view(np.float32)


def _to_dev(a, dtype):
    if dtype == "bf16":
        return to_dev_u16(a)
    if dtype == "f16":
        return to_dev_u16(np.asarray(a, np.float16).view(np.uint16)).view(torch.float16)
    return to_dev_f32(a)


def _bits(a):
    a = np.asarray(a)
    return a.view(np.uint16) if a.dtype.itemsize == 2 else a.view(np.uint32)


def _same(got, want):
    """Bit for bit, except that where the oracle holds a float NaN only the
    class is compared (a NaN's payload after an fp16 conversion is left open)."""
    got, want = np.asarray(got), np.asarray(want)
    if want.dtype in (np.float16, np.float32):
        nan = np.isnan(want)
        if nan.any():
            g = got.view(want.dtype)
            return bool(np.array_equal(np.isnan(g), nan)) and bool(np.array_equal(_bits(g)[~nan], _bits(want)[~nan]))
    return bool(np.array_equal(_bits(got), _bits(want)))


def _chunks(W, S, dtype, host=None):
    """W separately allocated chunks, optionally filled from a host [W*S] array."""
    cs = [Guarded(S, TORCH[dtype]) for _ in range(W)]
    if host is not None:
        for i, c in enumerate(cs):
            if S:
                c.view.copy_(_to_dev(host[i * S:(i + 1) * S], dtype))
    return cs


def _wide_f32(words, n):
    rng = np.random.default_rng(words)
    return (rng.standard_normal(n) * np.exp2(rng.integers(-30, 31, n))).astype(np.float32)


@pytest.mark.parametrize("case", range(len(CASES)))
@pytest.mark.parametrize("align", [8, 1])
def test_ex_small(case, align, max_workgroups=0):
    W, dims = CASES[case]
    plan = BucketPlan(W, dims, align, max_workgroups=max_workgroups)
    oplan = O.make_plan(W, dims, align)
    S = oplan.chunk
    P = len(dims)
    for shift in (0, 1):
        # ---- ag_pack_ex, fp32 and bf16
        for r in sorted({0, W // 2, W - 1}):
            shards = [random_bits32([case, r, p, 1], O.local_elems(oplan, p, r)).view(np.float32) for p in range(P)]
            bufs = [Guarded(s.size, torch.float32, shift) for s in shards]
            for b, s in zip(bufs, shards):
                if s.size:
                    b.view.copy_(to_dev_f32(s))
            for dtype in ("f32", "bf16", "f16"):
                out = Guarded(S, TORCH[dtype])
                step(f"ag_pack_ex {dtype} W={W} case={case} rank={r} align={align} shift={shift}")
                plan.ag_pack_ex(r, [b.view for b in bufs], out.view, dtype)
                torch.cuda.synchronize()
                assert out.guards_intact()
                want = O.ag_pack(oplan, r, shards, dtype)
                assert _same(_host(out.view, dtype), want if dtype != "bf16" else _bits(want))
        # ---- ag_unpack_ex from W separate chunks
        for dtype in ("bf16", "f32", "f16"):
            if dtype == "f32":
                g = random_bits32([case, 3], W * S).view(np.float32)
            else:
                g = random_bits16([case, 2], W * S)
                if dtype == "f16":
                    g = g.view(np.float16)
            chunks = _chunks(W, S, dtype, g)
            outs = [Guarded(n * k, TORCH[dtype], shift) for n, k in dims]
            step(f"ag_unpack_ex {dtype} W={W} case={case} align={align} shift={shift}")
            plan.ag_unpack_ex([c.view for c in chunks], [o.view for o in outs], dtype)
            torch.cuda.synchronize()
            want = O.ag_unpack(oplan, g)
            for p, o in enumerate(outs):
                assert o.guards_intact(), p
                assert np.array_equal(_bits(_host(o.view, dtype)), _bits(want[p].reshape(-1))), (dtype, p)
        # ---- rs_pack_ex into W separate chunks: bf16->bf16, bf16->f32, f32->f32
        for gdt, wire in (("bf16", "bf16"), ("bf16", "f32"), ("f32", "f32"), ("f16", "f16"), ("f16", "f32")):
            if gdt == "bf16":
                grads = [random_bits16([case, 4, p], n * k) for p, (n, k) in enumerate(dims)]
            elif gdt == "f16":
                grads = [random_bits16([case, 8, p], n * k).view(np.float16) for p, (n, k) in enumerate(dims)]
            else:
                grads = [random_bits32([case, 5, p], n * k).view(np.float32) for p, (n, k) in enumerate(dims)]
            gbufs = [Guarded(gg.size, TORCH[gdt], shift) for gg in grads]
            for b, gg in zip(gbufs, grads):
                if gg.size:
                    b.view.copy_(_to_dev(gg, gdt))
            chunks = _chunks(W, S, wire)
            step(f"rs_pack_ex {gdt}->{wire} W={W} case={case} align={align} shift={shift}")
            plan.rs_pack_ex([b.view for b in gbufs], [c.view for c in chunks], wire)
            torch.cuda.synchronize()
            want = O.rs_pack(oplan, [gg.reshape(n, k) for gg, (n, k) in zip(grads, dims)],
                             None if gdt == wire else wire)
            for j, c in enumerate(chunks):
                assert c.guards_intact(), j
                assert _same(_host(c.view, wire), want[j * S:(j + 1) * S]), (gdt, wire, j)
        # ---- rs_reduce_ex from W separate chunks, bf16 and f32
        for dtype in ("bf16", "f32", "f16"):
            if dtype == "bf16":
                rng = np.random.default_rng([case, 6])
                recv = ((rng.standard_normal(W * S) * np.exp2(rng.integers(-20, 21, W * S)))
                        .astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
            elif dtype == "f16":
                rng = np.random.default_rng([case, 9])
                recv = (rng.integers(0, 0x7C00, W * S) | (rng.integers(0, 2, W * S) << 15)).astype(np.uint16)
                recv = recv.view(np.float16)
            else:
                recv = _wide_f32([case, 7], W * S)
            chunks = _chunks(W, S, dtype, recv)
            for r in sorted({0, W - 1}):
                outs = [Guarded(O.local_elems(oplan, p, r), torch.float32, shift) for p in range(P)]
                step(f"rs_reduce_ex {dtype} W={W} case={case} rank={r} align={align} shift={shift}")
                plan.rs_reduce_ex(r, [c.view for c in chunks], [o.view for o in outs], dtype)
                torch.cuda.synchronize()
                want = O.rs_reduce(oplan, r, recv)
                for p, o in enumerate(outs):
                    assert o.guards_intact(), p
                    assert np.array_equal(host_u32(o.view), want[p].reshape(-1).view(np.uint32)), (dtype, r, p)
    plan.close()


@pytest.mark.parametrize("case", range(len(CASES)))
def test_ag_pack_push(case, max_workgroups=0):
    """The packed chunk of one rank written to W separate destinations, bf16
    and fp32: every destination equals the oracle's pack."""
    W, dims = CASES[case]
    for align in (8, 1):
        plan = BucketPlan(W, dims, align, max_workgroups=max_workgroups)
        oplan = O.make_plan(W, dims, align)
        S = oplan.chunk
        P = len(dims)
        for r in sorted({0, W - 1}):
            shards = [random_bits32([case, r, p, 11], O.local_elems(oplan, p, r)).view(np.float32) for p in range(P)]
            bufs = [Guarded(s_.size, torch.float32, r % 2) for s_ in shards]
            for b, s_ in zip(bufs, shards):
                if s_.size:
                    b.view.copy_(to_dev_f32(s_))
            for dtype in ("bf16", "f32", "f16"):
                dsts = _chunks(W, S, dtype)
                step(f"ag_pack_push {dtype} W={W} case={case} rank={r} align={align}")
                plan.ag_pack_push(r, [b.view for b in bufs], [d.view for d in dsts], dtype)
                torch.cuda.synchronize()
                want = O.ag_pack(oplan, r, shards, dtype)
                for j, d in enumerate(dsts):
                    assert d.guards_intact(), j
                    assert _same(_host(d.view, dtype), want), (dtype, j)
        plan.close()


@pytest.mark.parametrize("W", [15, 16, 17, 18, 33, 34])
def test_push_destination_rows(W):
    """The copy half of the push around its row size of 16 destinations:
    W - 1 = 14 and 15 take one row of every destination, 16 one full row,
    17 a full row and a row of one, 32 two full rows, 33 two and a row of
    one; the source rank at either end and inside a row.  Chunks of a few
    2 KB tiles, whole (align 8) and with a partial 16-byte unit (align 1)."""
    dims = [(600 * W + 7, 5), (2, 3), (W, 1)]
    for align in (8, 1):
        plan = BucketPlan(W, dims, align)
        oplan = O.make_plan(W, dims, align)
        S = oplan.chunk
        for r in sorted({0, 5, W // 2, W - 1}):
            shards = [random_bits32([W, r, p, 13], O.local_elems(oplan, p, r)).view(np.float32)
                      for p in range(len(dims))]
            dsts = _chunks(W, S, "bf16")
            step(f"ag_pack_push bf16 W={W} rank={r} align={align}")
            plan.ag_pack_push(r, [to_dev_f32(s_) for s_ in shards], [d.view for d in dsts])
            torch.cuda.synchronize()
            want = O.ag_pack(oplan, r, shards, "bf16")
            for j, d in enumerate(dsts):
                assert d.guards_intact(), j
                assert _same(_host(d.view, "bf16"), want), j
        plan.close()


@pytest.mark.parametrize("cap", [1, 7])
def test_ex_grid_stride(cap):
    """The element-type and chunk-table forms with every workgroup looping over
    many tiles."""
    test_ex_small(5, 8, max_workgroups=cap)


@pytest.mark.parametrize("cap", [1, 7, 50])
def test_push_grid_stride(cap):
    """The push at W = 48 (a pack and a copy) with every workgroup looping over
    many work items, including caps that are not a multiple of the XCD count."""
    assert CASES[4][0] == 48
    test_ag_pack_push(4, max_workgroups=cap)


def test_ex_chunks_alias_one_buffer():
    """The chunk table may point into one [W][S] buffer: the results equal the
    contiguous calls bit for bit."""
    wl = WORKLOADS[1]
    W = wl.world_size
    plan = BucketPlan(W, wl.dims)
    S = plan.chunk_elems
    gathered = dev_random_bits16(W * S, 71)
    a = [torch.empty(n * k, dtype=torch.bfloat16, device=DEV) for n, k in wl.dims]
    b = [torch.empty(n * k, dtype=torch.bfloat16, device=DEV) for n, k in wl.dims]
    step("ag_unpack contiguous vs chunk table")
    plan.ag_unpack(gathered, a)
    plan.ag_unpack_ex([gathered[i * S:(i + 1) * S] for i in range(W)], b)
    oa = [torch.empty(plan.local_elems(p, 1), device=DEV) for p in range(len(wl.dims))]
    ob = [torch.empty(plan.local_elems(p, 1), device=DEV) for p in range(len(wl.dims))]
    plan.rs_reduce(1, gathered, oa)
    plan.rs_reduce_ex(1, [gathered[i * S:(i + 1) * S] for i in range(W)], ob)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    for x, y in zip(oa, ob):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))


@pytest.mark.parametrize("key", [3])
def test_ex_workload_full(key):
    """The 70B block (W = 64) at full size: fp32 wire and chunk tables."""
    wl = WORKLOADS[key]
    W = wl.world_size
    plan = BucketPlan(W, wl.dims)
    oplan = O.make_plan(W, wl.dims)
    S = oplan.chunk
    P = wl.num_params
    # fp32 param_dtype pack of rank 0 and W-1
    for r in (0, W - 1):
        shards = [random_bits32([key, r, p, 9], O.local_elems(oplan, p, r)).view(np.float32) for p in range(P)]
        out = Guarded(S, torch.float32)
        step(f"ag_pack_ex f32 full W={W} rank={r}")
        plan.ag_pack_ex(r, [to_dev_f32(s) for s in shards], out.view, "f32")
        torch.cuda.synchronize()
        assert out.guards_intact()
        assert np.array_equal(host_u32(out.view), O.ag_pack(oplan, r, shards, "f32").view(np.uint32))
    # the fp16 pack of rank W-1
    r = W - 1
    shards = [random_bits32([key, r, p, 13], O.local_elems(oplan, p, r)).view(np.float32) for p in range(P)]
    out = Guarded(S, torch.float16)
    step(f"ag_pack_ex f16 full W={W} rank={r}")
    plan.ag_pack_ex(r, [to_dev_f32(s_) for s_ in shards], out.view, "f16")
    torch.cuda.synchronize()
    assert out.guards_intact()
    assert _same(_host(out.view, "f16"), O.ag_pack(oplan, r, shards, "f16"))
    # the bf16 pack of rank 1 pushed to all W gathered buffers
    r = 1
    shards = [random_bits32([key, r, p, 12], O.local_elems(oplan, p, r)).view(np.float32) for p in range(P)]
    dsts = [torch.empty(S, dtype=torch.bfloat16, device=DEV) for _ in range(W)]
    step(f"ag_pack_push bf16 full W={W} rank={r}")
    plan.ag_pack_push(r, [to_dev_f32(s_) for s_ in shards], dsts)
    torch.cuda.synchronize()
    want = O.ag_pack(oplan, r, shards)
    for j in range(W):
        assert np.array_equal(host_u16(dsts[j]), want), j
    del dsts, want
    # bf16 gradients cast to an fp32 wire, pushed into W chunks
    grads = [dev_random_bits16(n * k, 300 + p) for p, (n, k) in enumerate(wl.dims)]
    chunks = [torch.empty(S, dtype=torch.float32, device=DEV) for _ in range(W)]
    step(f"rs_pack_ex bf16->f32 full W={W}")
    plan.rs_pack_ex(grads, chunks, "f32")
    torch.cuda.synchronize()
    want = O.rs_pack(oplan, [host_u16(g).reshape(n, k) for g, (n, k) in zip(grads, wl.dims)], "f32")
    for j in range(W):
        assert np.array_equal(host_u32(chunks[j]), want[j * S:(j + 1) * S].view(np.uint32)), j
    del grads, want
    # fp32 reduce of rank 0 pulling W chunks
    recv = [dev_wide_f32(S, 800 + i) for i in range(W)]
    outs = [torch.empty(O.local_elems(oplan, p, 0), dtype=torch.float32, device=DEV) for p in range(P)]
    step(f"rs_reduce_ex f32 full W={W}")
    plan.rs_reduce_ex(0, recv, outs, "f32")
    torch.cuda.synchronize()
    want = O.rs_reduce(oplan, 0, np.concatenate([host_u32(c).view(np.float32) for c in recv]))
    for p in range(P):
        assert np.array_equal(host_u32(outs[p]), want[p].reshape(-1).view(np.uint32)), p
    plan.close()


@pytest.mark.parametrize("key,align", [(2, 8), (5, 1), (7, 8), (4, 8)])
def test_push_workload_full(key, align):
    """The push at full size on the other large buckets: the single-row copy
    (the 8B block, W = 8) and the copy in rows of 16 (the uneven bucket,
    W = 48, densely packed so that its chunk ends in a partial 16-byte unit;
    the 8B block at W = 128; the 405B block, W = 128).  The source rank's
    chunk is compared with the oracle's pack; every other destination must
    equal it bit for bit (compared on the device)."""
    wl = WORKLOADS[key]
    W = wl.world_size
    plan = BucketPlan(W, wl.dims, align)
    oplan = O.make_plan(W, wl.dims, align)
    S = oplan.chunk
    P = wl.num_params
    r = W - 1 if key == 5 else W // 2
    shards = [random_bits32([key, r, p, 14], O.local_elems(oplan, p, r)).view(np.float32) for p in range(P)]
    dsts = [torch.empty(S, dtype=torch.bfloat16, device=DEV) for _ in range(W)]
    for d in dsts:
        d.view(torch.int16).fill_(-1)
    step(f"ag_pack_push bf16 full {wl.name} W={W} rank={r} align={align}")
    plan.ag_pack_push(r, [to_dev_f32(s_) for s_ in shards], dsts)
    torch.cuda.synchronize()
    assert np.array_equal(host_u16(dsts[r]), O.ag_pack(oplan, r, shards))
    src = dsts[r].view(torch.int16)
    for j in range(W):
        assert torch.equal(dsts[j].view(torch.int16), src), j
    del dsts
    plan.close()
    torch.cuda.empty_cache()


def test_ex_workload_full_chunk_tables():
    """The 70B block (W = 64) at full size through the W-pointer forms the
    benchmark times: unpack pulling W chunks, rs_pack pushing into W chunks,
    and the bf16 and fp16 reduces pulling W chunks."""
    wl = WORKLOADS[3]
    W = wl.world_size
    plan = BucketPlan(W, wl.dims)
    oplan = O.make_plan(W, wl.dims)
    S = oplan.chunk
    P = wl.num_params
    # unpack from W chunks of random bf16 bit patterns
    chunks = [dev_random_bits16(S, 900 + i) for i in range(W)]
    params = [torch.empty(n * k, dtype=torch.bfloat16, device=DEV) for n, k in wl.dims]
    step(f"ag_unpack_ex bf16 chunks full W={W}")
    plan.ag_unpack_ex(chunks, params, "bf16")
    torch.cuda.synchronize()
    want = O.ag_unpack(oplan, np.concatenate([host_u16(c) for c in chunks]))
    for p in range(P):
        assert np.array_equal(host_u16(params[p]), want[p].reshape(-1)), p
    del chunks, want
    # rs_pack of the block's gradients into W chunks
    grads = [dev_random_bits16(n * k, 950 + p) for p, (n, k) in enumerate(wl.dims)]
    dsts = [torch.empty(S, dtype=torch.bfloat16, device=DEV) for _ in range(W)]
    step(f"rs_pack_ex bf16 chunks full W={W}")
    plan.rs_pack_ex(grads, dsts, "bf16")
    torch.cuda.synchronize()
    want = O.rs_pack(oplan, [host_u16(g).reshape(n, k) for g, (n, k) in zip(grads, wl.dims)])
    for j in range(W):
        assert np.array_equal(host_u16(dsts[j]), want[j * S:(j + 1) * S]), j
    del grads, dsts, want, params
    # bf16 reduce of rank W-1 from W chunks
    recv = [dev_wide_bf16(S, 1000 + i) for i in range(W)]
    outs = [torch.empty(O.local_elems(oplan, p, W - 1), dtype=torch.float32, device=DEV) for p in range(P)]
    step(f"rs_reduce_ex bf16 chunks full W={W} rank={W - 1}")
    plan.rs_reduce_ex(W - 1, recv, outs, "bf16")
    torch.cuda.synchronize()
    want = O.rs_reduce(oplan, W - 1, np.concatenate([host_u16(c) for c in recv]))
    for p in range(P):
        assert np.array_equal(host_u32(outs[p]), want[p].reshape(-1).view(np.uint32)), p
    del recv, outs, want
    # fp16 reduce of rank 0: finite fp16 values (exponent field below 16), W chunks
    recv = [dev_random_bits16(S, 1100 + i) for i in range(W)]
    for c in recv:
        c.view(torch.int16).bitwise_and_(-0x4001)      # 0xBFFF: clears the exponent's top bit
    outs = [torch.empty(O.local_elems(oplan, p, 0), dtype=torch.float32, device=DEV) for p in range(P)]
    step(f"rs_reduce_ex f16 chunks full W={W} rank=0")
    plan.rs_reduce_ex(0, [c.view(torch.float16) for c in recv], outs, "f16")
    torch.cuda.synchronize()
    want = O.rs_reduce(oplan, 0, np.concatenate([host_u16(c) for c in recv]).view(np.float16))
    for p in range(P):
        assert np.array_equal(host_u32(outs[p]), want[p].reshape(-1).view(np.uint32)), p
    plan.close()
    torch.cuda.empty_cache()

