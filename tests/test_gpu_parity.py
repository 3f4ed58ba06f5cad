"""GPU parity: every kernel, through the C ABI, against the CPU oracle, bit for bit.

Outputs live inside poisoned guard bands: every output element must equal the
oracle's (so nothing is left unwritten) and the guards must be intact (so
nothing is written out of bounds).  Small buckets cover the edge cases (empty
parameters, ranks holding no rows, W = 1, dim 0 smaller than W, 1-wide
parameters, the dense align = 1 layout, element-aligned parameter pointers,
the parameter limit, several tiles with ragged tails); the Llama-shaped
workloads, the 405B block included, run at full size in the launch
configuration the benchmark times, with every output element compared, at
ranks 0, W/2 and W-1 for the per-rank kernels.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle.fsdp_oracle as O
from gpu_util import (DEV, Guarded, dev_random_bits16, dev_random_f32_bits, dev_wide_bf16, host_u16,
                      host_u32, step, to_dev_f32, to_dev_u16)
from synth import WORKLOADS, random_bits16, random_bits32

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

if torch.cuda.is_available():
    from paper_2411_00284_amd import BucketPlan


SMALL = [
    (1, [(5, 3), (1, 1), (0, 4)]),
    (2, [(5, 3), (1, 1), (7, 2), (0, 4)]),
    (3, [(7, 3), (2, 5), (10, 1), (3, 8)]),
    (4, [(16, 8), (9, 3), (3, 1), (4, 16), (1, 7)]),
    (7, [(20, 2), (6, 1), (13, 9)]),
    (8, [(17, 8), (8, 8), (64, 1), (1, 1)]),
    (48, [(86, 1), (4096, 1), (1, 3), (47, 2), (49, 1)]),
    (64, [(65, 1), (128, 2), (0, 3)]),
    # several tiles per segment, ragged tails, unaligned segment lengths
    (3, [(5000, 7), (4096, 4), (1, 1), (20000, 1), (2049, 8)]),
    (5, [(40000, 3), (9, 4096)]),
    # the parameter limit
    (4, [(i % 13, 1 + i % 5) for i in range(64)]),
    # one large and many tiny parameters (the pack kernel's tile-lookup grid)
    (2, [(200000, 1)] + [(1, 1)] * 8),
]


def _ranks(w):
    return sorted({0, w // 2, w - 1})


# ----------------------------------------------------------------- one kernel each

def run_ag_pack(plan, oplan, rank, seed, shift=0):
    """Random fp32 bit patterns (NaN, inf, subnormals) as the rank's shards."""
    P = oplan.num_params
    host = [random_bits32([seed, rank, p], O.local_elems(oplan, p, rank)).view(np.float32) for p in range(P)]
    bufs = [Guarded(h.size, torch.float32, shift) for h in host]
    for b, h in zip(bufs, host):
        if h.size:
            b.view.copy_(to_dev_f32(h))
    out = Guarded(oplan.chunk, torch.bfloat16)
    step(f"ag_pack W={oplan.world_size} P={P} rank={rank} align={oplan.align} shift={shift}")
    plan.ag_pack(rank, [b.view for b in bufs], out.view)
    torch.cuda.synchronize()
    assert out.guards_intact()
    assert np.array_equal(host_u16(out.view), O.ag_pack(oplan, rank, host))


def run_ag_unpack(plan, oplan, seed, shift=0):
    W, S = oplan.world_size, oplan.chunk
    g = random_bits16([seed, 1], W * S)
    gathered = Guarded(W * S, torch.bfloat16)
    gathered.view.copy_(to_dev_u16(g))
    outs = [Guarded(n * k, torch.bfloat16, shift) for n, k in zip(oplan.rows, oplan.inner)]
    step(f"ag_unpack W={W} P={oplan.num_params} align={oplan.align} shift={shift}")
    plan.ag_unpack(gathered.view, [o.view for o in outs])
    torch.cuda.synchronize()
    want = O.ag_unpack(oplan, g)
    for p, o in enumerate(outs):
        assert o.guards_intact(), p
        assert np.array_equal(host_u16(o.view), want[p].reshape(-1)), p
    assert np.array_equal(host_u16(gathered.view), g)           # input untouched


def run_rs_pack(plan, oplan, seed, shift=0):
    W, S = oplan.world_size, oplan.chunk
    grads = [random_bits16([seed, 2, p], n * k) for p, (n, k) in enumerate(zip(oplan.rows, oplan.inner))]
    bufs = [Guarded(g.size, torch.bfloat16, shift) for g in grads]
    for b, g in zip(bufs, grads):
        if g.size:
            b.view.copy_(to_dev_u16(g))
    out = Guarded(W * S, torch.bfloat16)
    step(f"rs_pack W={W} P={oplan.num_params} align={oplan.align} shift={shift}")
    plan.rs_pack([b.view for b in bufs], out.view)
    torch.cuda.synchronize()
    assert out.guards_intact()
    want = O.rs_pack(oplan, [g.reshape(n, k) for g, n, k in zip(grads, oplan.rows, oplan.inner)])
    assert np.array_equal(host_u16(out.view), want)


def run_rs_reduce(plan, oplan, rank, recv_host, shift=0):
    W, S = oplan.world_size, oplan.chunk
    recv = Guarded(W * S, torch.bfloat16)
    recv.view.copy_(to_dev_u16(recv_host))
    outs = [Guarded(O.local_elems(oplan, p, rank), torch.float32, shift) for p in range(oplan.num_params)]
    step(f"rs_reduce W={W} P={oplan.num_params} rank={rank} align={oplan.align} shift={shift}")
    plan.rs_reduce(rank, recv.view, [o.view for o in outs])
    torch.cuda.synchronize()
    want = O.rs_reduce(oplan, rank, recv_host)
    for p, o in enumerate(outs):
        assert o.guards_intact(), p
        assert np.array_equal(host_u32(o.view), want[p].reshape(-1).view(np.uint32)), p


def wide_bf16_host(words, n):
    """Finite bf16 values over a wide exponent range (host copy of the same recipe)."""
    rng = np.random.default_rng(words)
    g = rng.standard_normal(n) * np.exp2(rng.integers(-20, 21, n))
    return (g.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


# ----------------------------------------------------------------- small buckets

@pytest.mark.parametrize("tiles", ["full", "half"])
def test_reduce_tile_sizes(tiles):
    """The reduction with its tile size forced each way (full-size tiles of 256
    threads, half-size tiles of 128) on the small buckets, which otherwise
    take the half-size tiles: every output bit for bit."""
    for case in range(len(SMALL)):
        w, dims = SMALL[case]
        plan = BucketPlan(w, dims, reduce_tiles=tiles)
        oplan = O.make_plan(w, dims)
        recv = wide_bf16_host([case, 77], w * oplan.chunk)
        for r in _ranks(w):
            run_rs_reduce(plan, oplan, r, recv)
        plan.close()


@pytest.mark.parametrize("cap", [1, 3, 50])
@pytest.mark.parametrize("case", [3, 8, 10, 11])
def test_grid_stride(case, cap):
    """With the workgroup cap lowered, every workgroup loops over many tiles
    (of several parameters, and through the reduce's LDS staging more than
    once); the results stay bit-exact."""
    w, dims = SMALL[case]
    plan = BucketPlan(w, dims, 8, max_workgroups=cap)
    oplan = O.make_plan(w, dims, 8)
    for r in _ranks(w):
        run_ag_pack(plan, oplan, r, seed=case)
    run_ag_unpack(plan, oplan, seed=case)
    run_rs_pack(plan, oplan, seed=case)
    recv = wide_bf16_host([case, cap], w * oplan.chunk)
    for r in _ranks(w):
        run_rs_reduce(plan, oplan, r, recv)
    plan.close()


@pytest.mark.parametrize("cap", [0, 1, 7, 300])
def test_copy_tile_runs(cap):
    """The copies deal their tiles to the dies in runs (groups of 8 runs,
    then a tail in plain order); a bucket of two whole groups and a tail,
    with and without a workgroup cap, copies every element exactly once."""
    w, dims = 8, [(2_000_000, 5), (4099, 3), (13, 1)]
    plan = BucketPlan(w, dims, 8, max_workgroups=cap)
    oplan = O.make_plan(w, dims, 8)
    tiles = w * sum(-(-L // 2048) for L in oplan.seg)
    assert 2 * 8 * 256 < tiles < 3 * 8 * 256                  # two whole groups and a tail
    run_ag_unpack(plan, oplan, seed=cap)
    run_rs_pack(plan, oplan, seed=cap)
    plan.close()


@pytest.mark.parametrize("cap", [0, 1, 7, 50])
@pytest.mark.parametrize("w,dims", [
    (1, [(8192 * 1050 + 5, 1), (3, 7), (1000, 37)]),
    (2, [(2000, 4096 * 2 + 8), (5, 3), (7777, 517)]),
])
def test_pack_big_tiles(w, dims, cap):
    """Buckets large enough for the single-chunk pack's big tiles (at least 4
    per CU), ragged at every parameter's end, with the grid as launched and
    with every workgroup looping over many big tiles."""
    cus = torch.cuda.get_device_properties(DEV).multi_processor_count
    oplan = O.make_plan(w, dims, 8)
    ends = list(oplan.offset[1:]) + [oplan.chunk]
    big_tiles = sum(-(-(e - o) // 8192) for o, e in zip(oplan.offset, ends))     # 256 threads x 4 x 8
    assert big_tiles >= 4 * cus
    plan = BucketPlan(w, dims, 8, max_workgroups=cap)
    for r in range(w):
        run_ag_pack(plan, oplan, r, seed=900 + cap)
    plan.close()


@pytest.mark.parametrize("case", range(len(SMALL)))
@pytest.mark.parametrize("align", [8, 1])
def test_small_buckets(case, align):
    w, dims = SMALL[case]
    plan = BucketPlan(w, dims, align)
    oplan = O.make_plan(w, dims, align)
    assert plan.chunk_elems == oplan.chunk
    for shift in (0, 1):
        for r in _ranks(w):
            run_ag_pack(plan, oplan, r, seed=case, shift=shift)
        run_ag_unpack(plan, oplan, seed=case, shift=shift)
        run_rs_pack(plan, oplan, seed=case, shift=shift)
        recv = wide_bf16_host([case, align], w * oplan.chunk)
        for r in _ranks(w):
            run_rs_reduce(plan, oplan, r, recv, shift=shift)
    plan.close()


def test_reduce_special_values():
    """Signed zeros, infinities, NaN and subnormals through the reduction."""
    w = 3
    dims = [(w * 40, 8)]
    plan = BucketPlan(w, dims)
    oplan = O.make_plan(w, dims)
    S = oplan.chunk
    specials = np.array([0x0000, 0x8000, 0x7F80, 0xFF80, 0x7FC0, 0x0001, 0x8001, 0x007F, 0x0080,
                         0x3F80, 0xBF80, 0x7F7F, 0xFF7F], np.uint16)
    rng = np.random.default_rng(5)
    recv = specials[rng.integers(0, specials.size, w * S)]
    recv[:S] = 0x8000                   # first rows: every source -0 -> -0
    recv[S:2 * S][:64] = 0x8000
    recv[2 * S:3 * S][:64] = 0x8000
    for r in range(w):
        run_rs_reduce(plan, oplan, r, recv)


def test_pack_special_values():
    """The fp32 -> bf16 cast on the hand-worked table and on every NaN class."""
    cases = [0x3F800000, 0x3F808000, 0x3F818000, 0x3F808001, 0x3F807FFF, 0x3F80FFFF, 0x3FFF8000,
             0x7F7FFFFF, 0x7F7F7FFF, 0x7F7F8000, 0x7F800000, 0xFF800000, 0x80000000, 0x00000000,
             0x00000001, 0x00008000, 0x00018000, 0x007FFFFF, 0x00400000, 0xBF808000, 0xBF818000,
             0x7FC00000, 0xFFC00000, 0x7F800001, 0xFF800001, 0x7FFFFFFF, 0xFFFFFFFF]
    x = np.array(cases * 40, np.uint32).view(np.float32)
    dims = [(x.size, 1)]
    plan = BucketPlan(1, dims)
    oplan = O.make_plan(1, dims)
    out = Guarded(oplan.chunk, torch.bfloat16)
    step("ag_pack special values")
    plan.ag_pack(0, [to_dev_f32(x)], out.view)
    torch.cuda.synchronize()
    assert out.guards_intact()
    assert np.array_equal(host_u16(out.view), O.ag_pack(oplan, 0, [x]))


def test_non_default_stream():
    w, dims = 4, [(300, 64), (7, 3)]
    plan = BucketPlan(w, dims)
    oplan = O.make_plan(w, dims)
    S = oplan.chunk
    g = random_bits16([77], w * S)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        gathered = to_dev_u16(g)
        outs = [torch.empty(n * k, dtype=torch.bfloat16, device=DEV) for n, k in dims]
        step("ag_unpack on a side stream")
        plan.ag_unpack(gathered, outs)            # enqueued on the current (side) stream
    s.synchronize()
    want = O.ag_unpack(oplan, g)
    for p in range(len(dims)):
        assert np.array_equal(host_u16(outs[p]), want[p].reshape(-1))


def test_repeat_calls_are_identical():
    """Poisoned outputs, two calls in a row: the second overwrites exactly as the first."""
    w, dims = 8, [(1000, 24), (33, 1)]
    plan = BucketPlan(w, dims)
    oplan = O.make_plan(w, dims)
    for _ in range(2):
        run_rs_pack(plan, oplan, seed=3)
        run_ag_pack(plan, oplan, 7, seed=3)


def test_plan_freed_while_launches_are_in_flight():
    """Kernel arguments are copied at launch: a plan freed right after the call
    returns (before the GPU has run the kernel) leaves the result intact."""
    w, dims = 8, [(20000, 64), (33, 1)]
    oplan = O.make_plan(w, dims)
    g = random_bits16([11, 1], w * oplan.chunk)
    gathered = to_dev_u16(g)
    outs = [torch.empty(n * k, dtype=torch.bfloat16, device=DEV) for n, k in dims]
    torch.cuda.synchronize()
    step("ag_unpack with the plan freed before the kernel runs")
    torch.cuda._sleep(10_000_000)                 # keep the stream busy so the launch waits
    plan = BucketPlan(w, dims)
    plan.ag_unpack(gathered, outs)
    plan.close()
    torch.cuda.synchronize()
    want = O.ag_unpack(oplan, g)
    for p, o in enumerate(outs):
        assert np.array_equal(host_u16(o), want[p].reshape(-1)), p


# ----------------------------------------------------------------- full-size workloads

def _full_ag_pack(plan, oplan, rank, seed):
    P = oplan.num_params
    shards = [dev_random_f32_bits(O.local_elems(oplan, p, rank), seed * 1000 + p) for p in range(P)]
    out = Guarded(oplan.chunk, torch.bfloat16)
    step(f"ag_pack full W={oplan.world_size} rank={rank}")
    plan.ag_pack(rank, shards, out.view)
    torch.cuda.synchronize()
    assert out.guards_intact()
    host = [host_u32(s).view(np.float32) for s in shards]
    assert np.array_equal(host_u16(out.view), O.ag_pack(oplan, rank, host))


def _full_ag_unpack(plan, oplan, seed):
    W, S = oplan.world_size, oplan.chunk
    gathered = dev_random_bits16(W * S, seed)
    outs = [Guarded(n * k, torch.bfloat16) for n, k in zip(oplan.rows, oplan.inner)]
    step(f"ag_unpack full W={W}")
    plan.ag_unpack(gathered, [o.view for o in outs])
    torch.cuda.synchronize()
    g = host_u16(gathered)
    want = O.ag_unpack(oplan, g)
    del g
    for p, o in enumerate(outs):
        assert o.guards_intact(), p
        assert np.array_equal(host_u16(o.view), want[p].reshape(-1)), p


def _full_rs_pack(plan, oplan, seed):
    W, S = oplan.world_size, oplan.chunk
    grads = [dev_random_bits16(n * k, seed * 100 + p) for p, (n, k) in enumerate(zip(oplan.rows, oplan.inner))]
    out = Guarded(W * S, torch.bfloat16)
    step(f"rs_pack full W={W}")
    plan.rs_pack(grads, out.view)
    torch.cuda.synchronize()
    assert out.guards_intact()
    host = [host_u16(g).reshape(n, k) for g, n, k in zip(grads, oplan.rows, oplan.inner)]
    del grads
    assert np.array_equal(host_u16(out.view), O.rs_pack(oplan, host))


def _full_rs_reduce(plan, oplan, rank, seed):
    W, S = oplan.world_size, oplan.chunk
    recv = dev_wide_bf16(W * S, seed)
    outs = [Guarded(O.local_elems(oplan, p, rank), torch.float32) for p in range(oplan.num_params)]
    step(f"rs_reduce full W={W} rank={rank}")
    plan.rs_reduce(rank, recv, [o.view for o in outs])
    torch.cuda.synchronize()
    want = O.rs_reduce(oplan, rank, host_u16(recv))
    for p, o in enumerate(outs):
        assert o.guards_intact(), p
        assert np.array_equal(host_u32(o.view), want[p].reshape(-1).view(np.uint32)), p


@pytest.mark.parametrize("key", [1, 2, 3, 5, 6, 7])
@pytest.mark.parametrize("kernel", ["ag_pack", "ag_unpack", "rs_pack", "rs_reduce"])
def test_workload_full(key, kernel):
    wl = WORKLOADS[key]
    plan = BucketPlan(wl.world_size, wl.dims)
    oplan = O.make_plan(wl.world_size, wl.dims)
    W = wl.world_size
    if kernel == "ag_pack":
        for r in _ranks(W):
            _full_ag_pack(plan, oplan, r, seed=key)
    elif kernel == "ag_unpack":
        _full_ag_unpack(plan, oplan, seed=key)
    elif kernel == "rs_pack":
        _full_rs_pack(plan, oplan, seed=key)
    else:
        for r in _ranks(W):
            _full_rs_reduce(plan, oplan, r, seed=key * 10 + r)
    plan.close()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("kernel", ["ag_pack", "ag_unpack", "rs_pack", "rs_reduce"])
def test_workload_uneven_dense(kernel):
    """The uneven bucket in the paper-literal dense layout (A = 1): the chunk
    stride S is odd, so the chunks of odd ranks and every segment after an
    odd-sized one start off the 16-byte grid (the misaligned vector paths);
    every output element at full size, ranks 0, W/2 and W-1."""
    wl = WORKLOADS[5]
    W = wl.world_size
    plan = BucketPlan(W, wl.dims, 1)
    oplan = O.make_plan(W, wl.dims, 1)
    assert plan.chunk_elems == oplan.chunk and oplan.chunk % 2 == 1
    if kernel == "ag_pack":
        for r in _ranks(W):
            _full_ag_pack(plan, oplan, r, seed=51)
    elif kernel == "ag_unpack":
        _full_ag_unpack(plan, oplan, seed=52)
    elif kernel == "rs_pack":
        _full_rs_pack(plan, oplan, seed=53)
    else:
        for r in _ranks(W):
            _full_rs_reduce(plan, oplan, r, seed=540 + r)
    plan.close()
    torch.cuda.empty_cache()


# ----------------------------------------------------------------- the 405B block, in full
#
# W = 128, W*S = 3.19e9 elements (64-bit indexing; 6.4 GB per bucket buffer).
# Every output element of every kernel is compared with the oracle; each
# kernel is a test of its own so that one test's host copies are freed before
# the next starts (about 20 GB of host memory at most).

W405 = WORKLOADS[4].world_size


def _plans_405b():
    wl = WORKLOADS[4]
    plan = BucketPlan(wl.world_size, wl.dims)
    oplan = O.make_plan(wl.world_size, wl.dims)
    assert plan.chunk_elems == oplan.chunk
    assert wl.world_size * oplan.chunk > 2 ** 31
    return plan, oplan


@pytest.mark.parametrize("rank", _ranks(W405))
def test_workload_405b_ag_pack(rank):
    plan, oplan = _plans_405b()
    _full_ag_pack(plan, oplan, rank, seed=4)
    plan.close()
    torch.cuda.empty_cache()


def test_workload_405b_ag_unpack():
    plan, oplan = _plans_405b()
    _full_ag_unpack(plan, oplan, seed=41)
    plan.close()
    torch.cuda.empty_cache()


def test_workload_405b_rs_pack():
    plan, oplan = _plans_405b()
    _full_rs_pack(plan, oplan, seed=42)
    plan.close()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("rank", _ranks(W405))
def test_workload_405b_rs_reduce(rank):
    plan, oplan = _plans_405b()
    _full_rs_reduce(plan, oplan, rank, seed=4200 + rank)
    plan.close()
    torch.cuda.empty_cache()
