"""The C-ABI library on the host (no GPU): exports, planner, argument checks.

The planner makes no HIP call, so the C++ plan is compared with the oracle's
plan here.  The error-path tests hand the library fake device addresses that
its host-side validation must reject before any HIP call; they run only where
no GPU is visible, so that a validation bug can never launch a kernel on them.
"""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import oracle.fsdp_oracle as O
from synth import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fsdp_bucket.h")

native = pytest.importorskip("paper_2411_00284_amd._native")
try:
    LIB = native.load()
except ImportError as e:  # pragma: no cover - the build step runs first
    pytest.fail(f"library not built: {e}")

from paper_2411_00284_amd import BucketPlan, FsdpError  # noqa: E402

no_gpu = pytest.mark.skipif(torch.cuda.device_count() > 0,
                            reason="fake device pointers are only used where no GPU can receive them")

OK, INVALID, ALIGN, OVERFLOW, TOO_MANY, NOMEM, HIP, OVERLAP = range(8)


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fsdp_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = header_functions()
    for required in ("fsdp_bucket_plan", "fsdp_ag_pack", "fsdp_ag_unpack", "fsdp_rs_pack", "fsdp_rs_reduce"):
        assert required in names


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", native.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    for name in header_functions():
        assert name in exported, name
        assert hasattr(LIB, name)
    assert set(native.SIGNATURES) == set(header_functions())


def test_header_compiles_as_c():
    src = '#include "fsdp_bucket.h"\nint main(void){fsdp_plan* p = 0; (void)p; return FSDP_OK;}\n'
    res = subprocess.run(["gcc", "-std=c99", "-x", "c", "-fsyntax-only", "-D__HIP_PLATFORM_AMD__",
                          f"-I{os.path.join(ROOT, 'include')}", "-I/opt/rocm/include", "-"],
                         input=src, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr


# ----------------------------------------------------------------- planner == oracle planner

def assert_plans_equal(w, dims, align):
    want = O.make_plan(w, dims, align)
    got = BucketPlan(w, [(n, k) for n, k in dims], align)
    assert got.chunk_elems == want.chunk
    for p in range(len(dims)):
        assert got.rows_per_rank(p) == want.rows_per_rank[p]
        assert got.offset(p) == want.offset[p]
        assert got.seg_elems(p) == want.seg[p]
        for r in sorted({0, 1 % w, w // 2, w - 1}):
            assert got.local_rows(p, r) == O.local_rows(want, p, r)
    got.close()


@pytest.mark.parametrize("key", sorted(WORKLOADS))
@pytest.mark.parametrize("align", [8, 1, 16])
def test_planner_matches_oracle_on_workloads(key, align):
    wl = WORKLOADS[key]
    assert_plans_equal(wl.world_size, wl.dims, align)


@settings(max_examples=200, deadline=None)
@given(w=st.sampled_from([1, 2, 3, 4, 7, 8, 48, 64, 128]),
       dims=st.lists(st.tuples(st.integers(0, 5000), st.sampled_from([1, 2, 3, 8, 4096])), min_size=1, max_size=64),
       align=st.sampled_from([1, 2, 4, 8, 16, 64]))
def test_planner_matches_oracle_random(w, dims, align):
    assert_plans_equal(w, dims, align)


def test_plan_shape_flattening():
    plan = BucketPlan(4, [(10, 3, 5), (7,), (0, 9)])
    assert plan.dims == [(10, 15), (7, 1), (0, 9)]
    want = O.make_plan(4, [(10, 15), (7, 1), (0, 9)])
    assert plan.chunk_elems == want.chunk


# ----------------------------------------------------------------- planner errors

def raw_plan(w, dims, align=8):
    n = len(dims)
    rows = (ctypes.c_int64 * max(n, 1))(*[d[0] for d in dims])
    inner = (ctypes.c_int64 * max(n, 1))(*[d[1] for d in dims])
    h = ctypes.c_void_p()
    st_ = LIB.fsdp_bucket_plan(w, n, rows, inner, align, ctypes.byref(h))
    return st_, h


@pytest.mark.parametrize("w,dims,align,code", [
    (0, [(4, 4)], 8, INVALID),
    (-3, [(4, 4)], 8, INVALID),
    (4, [], 8, INVALID),
    (4, [(-1, 4)], 8, INVALID),
    (4, [(4, 0)], 8, INVALID),
    (4, [(4, 4)], 3, INVALID),
    (4, [(4, 4)], 0, INVALID),
    (4, [(1, 1)] * 65, 8, TOO_MANY),
    (4, [(1 << 40, 1 << 30)], 8, OVERFLOW),
    (1 << 20, [(1 << 40, 1 << 10)] * 2, 8, OVERFLOW),
])
def test_planner_rejects(w, dims, align, code):
    st_, h = raw_plan(w, dims, align)
    assert st_ == code
    assert not h.value
    assert LIB.fsdp_last_error()


def raw_plan_ex(w, dims, options, align=8):
    n = len(dims)
    rows = (ctypes.c_int64 * n)(*[d[0] for d in dims])
    inner = (ctypes.c_int64 * n)(*[d[1] for d in dims])
    h = ctypes.c_void_p()
    opts = None if options is None else ctypes.byref(native.PlanOptions(*options))
    return LIB.fsdp_bucket_plan_ex(w, n, rows, inner, align, opts, ctypes.byref(h)), h


@pytest.mark.parametrize("options,code", [
    (None, OK),
    ((0, 0, 0), OK),
    ((7, 1, 0), OK),
    ((1, 2, 0), OK),
    ((-1, 0, 0), INVALID),
    ((0, 3, 0), INVALID),
    ((0, -1, 0), INVALID),
    ((0, 0, 1), INVALID),
])
def test_plan_options(options, code):
    """Launch options are checked at planning; a valid set gives the same plan."""
    st_, h = raw_plan_ex(4, [(5, 3), (8, 2)], options)
    assert st_ == code
    if code == OK:
        assert LIB.fsdp_plan_chunk_elems(h) == O.make_plan(4, [(5, 3), (8, 2)]).chunk
        LIB.fsdp_plan_free(h)
    else:
        assert not h.value
        assert LIB.fsdp_last_error()


def test_plan_options_in_the_binding():
    with pytest.raises(ValueError):
        BucketPlan(4, [(5, 3)], reduce_tiles="quarter")
    with pytest.raises(RuntimeError):
        BucketPlan(4, [(5, 3)], max_workgroups=-2)
    BucketPlan(4, [(5, 3)], max_workgroups=3, reduce_tiles="half").close()


def test_plan_queries_on_bad_input():
    st_, h = raw_plan(4, [(5, 3)])
    assert st_ == OK
    assert LIB.fsdp_plan_local_rows(h, 0, 4) == -1
    assert LIB.fsdp_plan_local_rows(h, 1, 0) == -1
    assert LIB.fsdp_plan_param(h, 1, None, None, None) == INVALID
    LIB.fsdp_plan_free(h)
    # a freed handle is unknown from then on
    assert LIB.fsdp_plan_chunk_elems(h) == -1
    assert LIB.fsdp_plan_world_size(h) == -1
    LIB.fsdp_plan_free(h)                      # double free is ignored
    LIB.fsdp_plan_free(None)
    assert LIB.fsdp_plan_chunk_elems(None) == -1


def test_status_strings():
    for code in range(8):
        assert LIB.fsdp_status_str(code)
    assert LIB.fsdp_status_str(99) == b"unknown status"


# ----------------------------------------------------------------- hot-call argument checks

FAKE = 1 << 40           # a 16-byte aligned address no test ever dereferences


def ptrs(*vals):
    return (ctypes.c_void_p * len(vals))(*vals)


@no_gpu
def test_hot_calls_reject_bad_arguments():
    st_, h = raw_plan(4, [(5, 3), (8, 2)])
    S = LIB.fsdp_plan_chunk_elems(h)
    assert st_ == OK and S > 0
    shards = ptrs(FAKE + 4096, FAKE + 8192)
    # unknown plan
    assert LIB.fsdp_ag_pack(ctypes.c_void_p(FAKE), 0, shards, FAKE, None) == INVALID
    # rank out of range
    assert LIB.fsdp_ag_pack(h, 4, shards, FAKE, None) == INVALID
    assert LIB.fsdp_ag_pack(h, -1, shards, FAKE, None) == INVALID
    assert LIB.fsdp_rs_reduce(h, 4, FAKE, shards, None) == INVALID
    # NULL pointer arrays and NULL buffers
    assert LIB.fsdp_ag_pack(h, 0, None, FAKE, None) == INVALID
    assert LIB.fsdp_ag_pack(h, 0, shards, None, None) == INVALID
    assert LIB.fsdp_ag_unpack(h, None, shards, None) == INVALID
    assert LIB.fsdp_rs_pack(h, shards, None, None) == INVALID
    assert LIB.fsdp_rs_reduce(h, 0, None, shards, None) == INVALID
    # a NULL parameter pointer where elements exist
    assert LIB.fsdp_ag_pack(h, 0, ptrs(FAKE + 4096, None), FAKE, None) == INVALID
    # bucket buffers must be 16-byte aligned
    assert LIB.fsdp_ag_pack(h, 0, shards, FAKE + 2, None) == ALIGN
    assert LIB.fsdp_ag_unpack(h, FAKE + 8, shards, None) == ALIGN
    assert LIB.fsdp_rs_pack(h, shards, FAKE + 4, None) == ALIGN
    assert LIB.fsdp_rs_reduce(h, 0, FAKE + 2, shards, None) == ALIGN
    # element alignment of parameter pointers
    assert LIB.fsdp_ag_pack(h, 0, ptrs(FAKE + 4098, FAKE + 8192), FAKE, None) == ALIGN
    assert LIB.fsdp_rs_pack(h, ptrs(FAKE + 4097, FAKE + 8192), FAKE + 65536, None) == ALIGN
    # overlap: output over an input, outputs over each other
    assert LIB.fsdp_ag_pack(h, 0, ptrs(FAKE + 16, FAKE + 8192), FAKE, None) == OVERLAP
    assert LIB.fsdp_ag_unpack(h, FAKE, ptrs(FAKE + 64, FAKE + 8192), None) == OVERLAP
    assert LIB.fsdp_ag_unpack(h, FAKE, ptrs(FAKE + 65536, FAKE + 65536 + 8), None) == OVERLAP
    assert LIB.fsdp_rs_pack(h, ptrs(FAKE + 4096, FAKE + 8192), FAKE + 4000, None) == OVERLAP
    assert LIB.fsdp_rs_reduce(h, 0, FAKE, ptrs(FAKE + 64, FAKE + 8192), None) == OVERLAP
    assert LIB.fsdp_rs_reduce(h, 0, FAKE, ptrs(FAKE + 65536, FAKE + 65536 + 4), None) == OVERLAP
    LIB.fsdp_plan_free(h)


@no_gpu
def test_valid_calls_reach_the_runtime():
    """Fully valid arguments (NULL allowed for parameters with no elements on
    the rank) pass every host check and reach the HIP runtime, which reports
    that there is no device here."""
    st_, h = raw_plan(4, [(1, 3), (0, 5)])
    assert st_ == OK
    # rank 1 holds no rows of either parameter
    assert LIB.fsdp_ag_pack(h, 1, ptrs(None, None), FAKE, None) == HIP
    assert LIB.fsdp_rs_reduce(h, 3, FAKE, ptrs(None, None), None) == OK     # nothing to write: no launch
    assert LIB.fsdp_rs_pack(h, ptrs(FAKE + 4096, None), FAKE, None) == HIP
    assert LIB.fsdp_ag_unpack(h, FAKE, ptrs(FAKE + 4096, None), None) == HIP
    LIB.fsdp_plan_free(h)


def test_binding_checks_tensors():
    plan = BucketPlan(2, [(4, 4)])
    with pytest.raises(ValueError):
        plan.ag_pack(0, [], torch.empty(plan.chunk_elems, dtype=torch.bfloat16))
    with pytest.raises(TypeError):
        plan.ag_pack(0, [torch.empty(8, dtype=torch.float64)], torch.empty(plan.chunk_elems, dtype=torch.bfloat16))
    with pytest.raises(ValueError):
        plan.ag_pack(0, [torch.empty(7)], torch.empty(plan.chunk_elems, dtype=torch.bfloat16))
    with pytest.raises(ValueError):     # host tensors are refused before the library is called
        plan.ag_pack(0, [torch.empty(8)], torch.empty(plan.chunk_elems, dtype=torch.bfloat16))
    with pytest.raises(FsdpError):
        BucketPlan(0, [(4, 4)])
    with pytest.raises(ValueError):
        BucketPlan(2, [()])
    plan.close()
    plan.close()


def test_binding_requires_one_device():
    """One call's tensors (and its stream, when it is a torch stream) must share
    a device: the kernels run on one device and dereference every pointer there."""
    from paper_2411_00284_amd.bucket import _check_device
    cpu, meta = torch.empty(3), torch.empty(3, device="meta")
    _check_device(None, [[cpu, None, torch.empty(0, device="meta")], [cpu]])   # empty tensors are not read
    _check_device(torch.device("cpu"), [[cpu], [cpu]])
    with pytest.raises(ValueError):
        _check_device(None, [[cpu], [meta]])
    with pytest.raises(ValueError):
        _check_device(torch.device("meta"), [[cpu]])


@no_gpu
def test_extended_calls_reject_bad_arguments():
    st_, h = raw_plan(4, [(5, 3), (8, 2)])
    assert st_ == OK
    shards = ptrs(FAKE + 4096, FAKE + 8192)
    chunks = ptrs(*[FAKE + (1 << 20) * (i + 1) for i in range(4)])
    outs = ptrs(FAKE + (1 << 24), FAKE + (1 << 24) + 4096)
    # unknown dtypes
    assert LIB.fsdp_ag_pack_ex(h, 0, shards, 7, FAKE, None) == INVALID
    assert LIB.fsdp_ag_unpack_ex(h, -1, chunks, outs, None) == INVALID
    assert LIB.fsdp_rs_pack_ex(h, 0, shards, 2, chunks, None) == INVALID
    assert LIB.fsdp_rs_reduce_ex(h, 0, 3, chunks, outs, None) == INVALID
    # a wire of another 16-bit type, or fp32 gradients on a 16-bit wire
    assert LIB.fsdp_rs_pack_ex(h, 1, shards, 0, chunks, None) == INVALID
    assert LIB.fsdp_rs_pack_ex(h, 1, shards, 2, chunks, None) == INVALID
    assert LIB.fsdp_rs_pack_ex(h, 0, shards, 2, chunks, None) == INVALID
    assert LIB.fsdp_rs_pack_ex(h, 2, shards, 0, chunks, None) == INVALID
    # NULL chunk table, NULL or misaligned chunk
    assert LIB.fsdp_ag_unpack_ex(h, 0, None, outs, None) == INVALID
    assert LIB.fsdp_rs_reduce_ex(h, 0, 0, ptrs(FAKE, FAKE + 64, None, FAKE + 192), outs, None) == INVALID
    assert LIB.fsdp_rs_reduce_ex(h, 0, 1, ptrs(FAKE, FAKE + 8, FAKE + 128, FAKE + 192), outs, None) == ALIGN
    # rank out of range
    assert LIB.fsdp_rs_reduce_ex(h, 4, 0, chunks, outs, None) == INVALID
    # output chunks must not overlap each other or the gradients
    assert LIB.fsdp_rs_pack_ex(h, 0, shards, 0, ptrs(FAKE, FAKE + 16, FAKE + 4096 * 8, FAKE + 4096 * 9),
                               None) == OVERLAP
    assert LIB.fsdp_rs_pack_ex(h, 0, ptrs(FAKE + (1 << 20) + 16, FAKE + 8192), 0, chunks, None) == OVERLAP
    # unpacked parameters must not overlap the chunks they are read from
    assert LIB.fsdp_ag_unpack_ex(h, 0, chunks, ptrs(FAKE + (1 << 20) + 16, FAKE + (1 << 24)), None) == OVERLAP
    # fp32 outputs need 4-byte alignment
    assert LIB.fsdp_ag_unpack_ex(h, 1, chunks, ptrs(FAKE + (1 << 24) + 2, FAKE + (1 << 25)), None) == ALIGN
    # the push: unknown dtype, NULL table, overlapping destinations, a destination over a shard
    assert LIB.fsdp_ag_pack_push(h, 0, shards, 5, chunks, None) == INVALID
    assert LIB.fsdp_ag_pack_push(h, 0, shards, 0, None, None) == INVALID
    assert LIB.fsdp_ag_pack_push(h, 4, shards, 0, chunks, None) == INVALID
    assert LIB.fsdp_ag_pack_push(h, 0, shards, 0, ptrs(FAKE, FAKE + 16, FAKE + 4096 * 8, FAKE + 4096 * 9),
                                 None) == OVERLAP
    assert LIB.fsdp_ag_pack_push(h, 0, ptrs(FAKE + (1 << 20) + 16, FAKE + 8192), 0, chunks, None) == OVERLAP
    assert LIB.fsdp_ag_pack_push(h, 0, shards, 1, ptrs(FAKE, FAKE + 8, FAKE + 4096, FAKE + 8192), None) == ALIGN
    LIB.fsdp_plan_free(h)
    # more chunks than the table holds
    st_, h = raw_plan(129, [(300, 2)])
    assert st_ == OK
    many = ptrs(*[FAKE + 4096 * i for i in range(129)])
    assert LIB.fsdp_ag_pack_push(h, 0, ptrs(FAKE + (1 << 30)), 0, many, None) == TOO_MANY
    assert LIB.fsdp_rs_reduce_ex(h, 0, 0, many, ptrs(FAKE + (1 << 30)), None) == TOO_MANY
    assert LIB.fsdp_ag_unpack_ex(h, 0, many, ptrs(FAKE + (1 << 30)), None) == TOO_MANY
    LIB.fsdp_plan_free(h)


@no_gpu
def test_extended_valid_calls_reach_the_runtime():
    st_, h = raw_plan(2, [(5, 3)])
    assert st_ == OK
    chunks = ptrs(FAKE, FAKE + 4096)
    assert LIB.fsdp_ag_pack_ex(h, 0, ptrs(FAKE + 65536), 1, FAKE, None) == HIP
    assert LIB.fsdp_ag_unpack_ex(h, 1, chunks, ptrs(FAKE + 65536), None) == HIP
    assert LIB.fsdp_rs_pack_ex(h, 0, ptrs(FAKE + 65536), 1, chunks, None) == HIP
    assert LIB.fsdp_rs_reduce_ex(h, 1, 1, chunks, ptrs(FAKE + 65536), None) == HIP
    assert LIB.fsdp_ag_pack_push(h, 1, ptrs(FAKE + 65536), 0, chunks, None) == HIP
    # fp16: the pack, the copy and widening packs, the reduce
    assert LIB.fsdp_ag_pack_ex(h, 0, ptrs(FAKE + 65536), 2, FAKE, None) == HIP
    assert LIB.fsdp_ag_unpack_ex(h, 2, chunks, ptrs(FAKE + 65536), None) == HIP
    assert LIB.fsdp_rs_pack_ex(h, 2, ptrs(FAKE + 65536), 2, chunks, None) == HIP
    assert LIB.fsdp_rs_pack_ex(h, 2, ptrs(FAKE + 65536), 1, chunks, None) == HIP
    assert LIB.fsdp_rs_reduce_ex(h, 1, 2, chunks, ptrs(FAKE + 65536), None) == HIP
    LIB.fsdp_plan_free(h)


@no_gpu
def test_widening_pack_tile_count_overflow():
    """A bucket the planner accepts can still need more than 2^31 - 1 work tiles
    for the widening pack (half-size tiles): the call fails with
    FSDP_ERR_OVERFLOW before any HIP call."""
    n = 2 * ((1 << 40) + 8)
    st_, h = raw_plan(2, [(n, 1)])
    assert st_ == OK
    chunks = ptrs(FAKE, FAKE + (1 << 44))
    assert LIB.fsdp_rs_pack_ex(h, 0, ptrs(FAKE + (1 << 46)), 1, chunks, None) == OVERFLOW
    assert b"tiles" in LIB.fsdp_last_error()
    LIB.fsdp_plan_free(h)


def test_last_error_is_per_thread():
    """Each thread reads the detail of its own last failed call."""
    import threading
    results = {}

    def worker(i):
        h = ctypes.c_void_p()
        rows = (ctypes.c_int64 * 1)(4)
        inner = (ctypes.c_int64 * 1)(4)
        msgs = []
        for _ in range(200):
            if i % 2:
                st_ = LIB.fsdp_bucket_plan(0, 1, rows, inner, 8, ctypes.byref(h))        # bad W
            else:
                st_ = LIB.fsdp_bucket_plan(4, 1, rows, inner, 3, ctypes.byref(h))        # bad align
            msgs.append((st_, LIB.fsdp_last_error()))
        results[i] = msgs

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(8)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    for i, msgs in results.items():
        want = b"world_size" if i % 2 else b"power of two"
        assert all(st_ == INVALID and want in m for st_, m in msgs), i


def test_plans_from_many_threads():
    """Plans created, queried and freed concurrently agree with the oracle."""
    import threading
    errors = []

    def worker(i):
        try:
            for k in range(50):
                w = 1 + (i * 7 + k) % 64
                dims = [(1 + (i + k) % 300, 1 + k % 5), (k % 17, 3)]
                want = O.make_plan(w, dims, 8)
                got = BucketPlan(w, dims, 8)
                assert got.chunk_elems == want.chunk
                got.close()
        except Exception as e:   # noqa: BLE001 - reported below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(8)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
