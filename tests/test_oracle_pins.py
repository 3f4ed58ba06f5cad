"""The CPU oracle against what the paper and the mathematics fix (no GPU).

Every check in ``oracle_checks`` runs against the oracle and must pass; then
each deliberately broken copy of the oracle (a plausible implementation
mistake planted on the CPU) must be caught by at least one check.
"""

from types import SimpleNamespace

import numpy as np
import pytest

import oracle.fsdp_oracle as O
import oracle_checks as C
from synth import WORKLOADS

SMALL_CASES = [
    (1, [(5, 3), (1, 1), (0, 4)]),
    (2, [(5, 3), (1, 1), (7, 2), (0, 4)]),
    (3, [(7, 3), (2, 5), (10, 1), (3, 8)]),
    (4, [(16, 8), (9, 3), (3, 1), (4, 16), (1, 7)]),
    (7, [(20, 2), (6, 1), (13, 9)]),
    (8, [(17, 8), (8, 8), (64, 1), (1, 1)]),
    (48, [(86, 1), (4096, 1), (1, 3), (47, 2), (49, 1)]),
    (64, [(65, 1), (128, 2)]),
]


def oracle_impl():
    return SimpleNamespace(
        make_plan=O.make_plan, local_rows=O.local_rows, bf16_rne=O.bf16_rne, f16_rne=O.f16_rne,
        ag_pack=O.ag_pack, ag_unpack=O.ag_unpack, rs_pack=O.rs_pack, rs_reduce=O.rs_reduce)


def run_all_checks(impl, quick=False):
    C.check_bf16_hex_table(impl)
    C.check_bf16_nan(impl)
    C.check_bf16_vs_torch(impl, n=1 << 14 if quick else 1 << 18)
    C.check_bf16_nearest_even(impl, n=500 if quick else 4000)
    C.check_plan_toy_table(impl)
    C.check_plan_sharding_matches_torch_chunk(impl, SMALL_CASES)
    C.check_plan_invariants(impl, SMALL_CASES)
    C.check_plan_even_workloads(impl, [WORKLOADS[k] for k in (1, 2, 3, 4, 6, 7)])
    for w, dims in SMALL_CASES[:6]:
        for r in sorted({0, w // 2, w - 1}):
            C.check_ag_pack_bruteforce(impl, w, dims, r, seed=w)
        C.check_ag_unpack_bruteforce(impl, w, dims, seed=w)
        C.check_rs_pack_bruteforce(impl, w, dims, seed=w)
        C.check_roundtrip_library(impl, w, dims, seed=w)
        C.check_rs_pack_equals_ag_layout(impl, w, dims, seed=w)
        C.check_ag_then_rs_replicated(impl, w, dims, seed=w)
        C.check_rs_reduce_bruteforce(impl, w, dims, w - 1, seed=w)
        C.check_rs_reduce_bruteforce(impl, w, dims, 0, seed=w, exact=True)
    # dense (paper-literal) layout
    C.check_ag_pack_bruteforce(impl, 3, [(7, 3), (2, 5), (10, 1)], 1, seed=9, align=1)
    C.check_ag_unpack_bruteforce(impl, 3, [(7, 3), (2, 5), (10, 1)], seed=9, align=1)
    C.check_rs_pack_bruteforce(impl, 3, [(7, 3), (2, 5), (10, 1)], seed=9, align=1)
    C.check_rs_reduce_bruteforce(impl, 3, [(7, 3), (2, 5), (10, 1)], 2, seed=9, align=1)
    C.check_rs_reduce_closed_forms(impl)
    C.check_rs_reduce_not_reciprocal(impl)
    for w in (3, 48):
        C.check_rs_exact_mean_bound(impl, w, seed=1)
    if not quick:
        for w, dims in SMALL_CASES[6:]:
            C.check_ag_then_rs_replicated(impl, w, dims, seed=w)
            C.check_roundtrip_library(impl, w, dims, seed=w)


def test_oracle_passes_every_pin():
    run_all_checks(oracle_impl())


# ----------------------------------------------------------------- mutants

def _bf16_truncate(x):
    return (np.ascontiguousarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _bf16_ties_away(x):
    u = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    return (((u + 0x8000) >> 16) & 0xFFFF).astype(np.uint16)


def _plan_floor_rows(w, dims, align=8):
    plan = O.make_plan(w, dims, align)
    # rows per rank rounded down: loses the remainder rows of uneven tensors
    cpr = tuple(max(1, n // w) for n, _ in dims)
    seg = tuple(c * k for c, (_, k) in zip(cpr, dims))
    off, pos = [], 0
    for L in seg:
        pos = -(-pos // align) * align
        off.append(pos)
        pos += L
    return O.Plan(w, align, plan.rows, plan.inner, cpr, seg, tuple(off), -(-pos // align) * align)


def _reduce_reciprocal(plan, rank, recv):
    W, S = plan.world_size, plan.chunk
    out = []
    for p in range(plan.num_params):
        n, k, o = O.local_rows(plan, p, rank), plan.inner[p], plan.offset[p]
        v = n * k
        acc = O.bf16_to_f32(recv[o:o + v])
        for i in range(1, W):
            acc = np.add(acc, O.bf16_to_f32(recv[i * S + o:i * S + o + v]), dtype=np.float32)
        out.append(np.multiply(acc, np.float32(1.0 / W), dtype=np.float32).reshape(n, k))
    return out


def _reduce_from_plus_zero(plan, rank, recv):
    W, S = plan.world_size, plan.chunk
    out = []
    for p in range(plan.num_params):
        n, k, o = O.local_rows(plan, p, rank), plan.inner[p], plan.offset[p]
        v = n * k
        acc = np.zeros(v, np.float32)
        for i in range(W):
            acc = np.add(acc, O.bf16_to_f32(recv[i * S + o:i * S + o + v]), dtype=np.float32)
        out.append(np.divide(acc, np.float32(W), dtype=np.float32).reshape(n, k))
    return out


def _reduce_reverse_order(plan, rank, recv):
    W, S = plan.world_size, plan.chunk
    out = []
    for p in range(plan.num_params):
        n, k, o = O.local_rows(plan, p, rank), plan.inner[p], plan.offset[p]
        v = n * k
        acc = O.bf16_to_f32(recv[(W - 1) * S + o:(W - 1) * S + o + v])
        for i in range(W - 2, -1, -1):
            acc = np.add(acc, O.bf16_to_f32(recv[i * S + o:i * S + o + v]), dtype=np.float32)
        out.append(np.divide(acc, np.float32(W), dtype=np.float32).reshape(n, k))
    return out


def _reduce_wrong_source_stride(plan, rank, recv):
    W, S = plan.world_size, plan.chunk
    out = []
    for p in range(plan.num_params):
        n, k, o = O.local_rows(plan, p, rank), plan.inner[p], plan.offset[p]
        v = n * k
        # reads every source at the destination's own offset (rank*S) only
        acc = O.bf16_to_f32(recv[rank * S + o:rank * S + o + v]) * np.float32(W)
        out.append(np.divide(acc, np.float32(W), dtype=np.float32).reshape(n, k))
    return out


def _unpack_rank_minor(plan, gathered):
    W, S = plan.world_size, plan.chunk
    out = []
    for p in range(plan.num_params):
        n, k, o = plan.rows[p], plan.inner[p], plan.offset[p]
        full = np.empty((n, k), np.uint16)
        c = plan.rows_per_rank[p]
        for row in range(n):
            i, q = row % W, row // W          # transposed row -> (rank, row) map
            if q >= c:
                i, q = row // c, row % c
            full[row] = gathered[i * S + o + q * k:i * S + o + q * k + k]
        out.append(full)
    return out


def _pack_no_zero_fill(plan, rank, shards):
    send = np.full(plan.chunk, 0x1234, np.uint16)
    for p in range(plan.num_params):
        v = O.local_elems(plan, p, rank)
        send[plan.offset[p]:plan.offset[p] + v] = O.bf16_rne(np.asarray(shards[p]).reshape(-1))
    return send


def _rs_pack_reversed(plan, grads):
    send = O.rs_pack(plan, grads)
    W, S = plan.world_size, plan.chunk
    return send.reshape(W, S)[::-1].reshape(-1).copy()


def _rs_pack_off_by_one_row(plan, grads):
    W, S = plan.world_size, plan.chunk
    send = np.zeros(W * S, np.uint16)
    for p in range(plan.num_params):
        n, k, c, L, o = plan.rows[p], plan.inner[p], plan.rows_per_rank[p], plan.seg[p], plan.offset[p]
        padded = np.zeros(((W + 1) * c, k), np.uint16)
        padded[1:n + 1] = np.asarray(grads[p]).reshape(n, k)       # shifted by one row
        flat = padded.reshape(-1)
        for j in range(W):
            send[j * S + o:j * S + o + L] = flat[j * L:(j + 1) * L]
    return send


MUTANTS = {
    "bf16 truncation": dict(bf16_rne=_bf16_truncate),
    "bf16 ties away from zero": dict(bf16_rne=_bf16_ties_away),
    "floor rows per rank": dict(make_plan=_plan_floor_rows),
    "reduce by reciprocal": dict(rs_reduce=_reduce_reciprocal),
    "reduce from +0": dict(rs_reduce=_reduce_from_plus_zero),
    "reduce in reverse rank order": dict(rs_reduce=_reduce_reverse_order),
    "reduce one source only": dict(rs_reduce=_reduce_wrong_source_stride),
    "unpack transposed rows": dict(ag_unpack=_unpack_rank_minor),
    "pack leaves padding unwritten": dict(ag_pack=_pack_no_zero_fill),
    "rs_pack destinations reversed": dict(rs_pack=_rs_pack_reversed),
    "rs_pack rows shifted": dict(rs_pack=_rs_pack_off_by_one_row),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    impl = oracle_impl()
    for k, v in MUTANTS[name].items():
        setattr(impl, k, v)
    # a mutant of the bf16 cast also has to be used by the pack
    if "bf16_rne" in MUTANTS[name]:
        bf = MUTANTS[name]["bf16_rne"]

        def pack(plan, rank, shards, bf=bf):
            send = np.zeros(plan.chunk, np.uint16)
            for p in range(plan.num_params):
                v = O.local_elems(plan, p, rank)
                send[plan.offset[p]:plan.offset[p] + v] = bf(np.asarray(shards[p]).reshape(-1))
            return send
        impl.ag_pack = pack
    if "make_plan" in MUTANTS[name]:
        mp = MUTANTS[name]["make_plan"]
        impl.local_rows = lambda plan, p, r: min(plan.rows_per_rank[p], max(0, plan.rows[p] - r * plan.rows_per_rank[p]))
        impl.make_plan = mp
    with pytest.raises((AssertionError, ValueError)):
        run_all_checks(impl, quick=True)


# ----------------------------------------------------------------- sliced forms

@pytest.mark.parametrize("w,dims", SMALL_CASES[:6] + [(48, [(86, 1), (100, 3), (1, 8)])])
def test_sliced_forms_equal_full_forms(w, dims):
    """The sliced oracle entry points (used at full bucket sizes) agree with the
    full-buffer ones on every slice of small buckets."""
    from synth import random_bits16, random_bits32
    for align in (8, 1):
        plan = O.make_plan(w, dims, align)
        S = plan.chunk
        rng = np.random.default_rng(w)
        for r in sorted({0, w // 2, w - 1}):
            shards = [random_bits32([w, r, p], O.local_elems(plan, p, r)).view(np.float32)
                      for p in range(len(dims))]
            full = O.ag_pack(plan, r, shards)
            for _ in range(5):
                k0 = int(rng.integers(0, S + 1)); k1 = int(rng.integers(k0, S + 1))
                got = O.ag_pack_range(plan, r, lambda p, lo, hi: shards[p][lo:hi], k0, k1)
                assert np.array_equal(got, full[k0:k1])
        g = random_bits16([w, 7], w * S)
        unp = O.ag_unpack(plan, g)
        for p, (n, k) in enumerate(dims):
            rows = list(range(n))
            assert np.array_equal(O.ag_unpack_rows(plan, lambda s, c: g[s:s + c], p, rows), unp[p])
        grads = [random_bits16([w, 8, p], n * k).reshape(n, k) for p, (n, k) in enumerate(dims)]
        send = O.rs_pack(plan, grads)
        for j in range(w):
            for k0, k1 in ((0, S), (1, S - 1), (S // 3, S // 2)):
                if k0 > k1:
                    continue
                got = O.rs_pack_range(plan, lambda p, lo, hi: grads[p].reshape(-1)[lo:hi], j, k0, k1)
                assert np.array_equal(got, send[j * S + k0:j * S + k1])
        recv = random_bits16([w, 9], w * S)
        for r in sorted({0, w - 1}):
            red = O.rs_reduce(plan, r, recv)
            for p in range(len(dims)):
                v = O.local_elems(plan, p, r)
                got = O.rs_reduce_range(plan, r, lambda s, c: recv[s:s + c], p, 0, v)
                assert np.array_equal(got.view(np.uint32), red[p].reshape(-1).view(np.uint32))


# ----------------------------------------------------------------- fp32 wires

@pytest.mark.parametrize("w,dims", SMALL_CASES[:6] + [(48, [(86, 1), (100, 3), (1, 8)])])
def test_fp32_variants(w, dims):
    impl = oracle_impl()
    C.check_f32_param_roundtrip(impl, w, dims, seed=w)
    C.check_f32_wire_same_bits(impl, w, dims, seed=w)
    C.check_rs_reduce_bruteforce_f32(impl, w, dims, w - 1, seed=w)
    C.check_rs_reduce_bruteforce_f32(impl, w, dims, 0, seed=w, align=1)


def test_fp32_pins_catch_a_rounding_pack():
    """A pack that rounds to bf16 and widens back when asked for fp32 fails."""
    impl = oracle_impl()

    def rounding_pack(plan, rank, shards, param_dtype="bf16"):
        send = O.ag_pack(plan, rank, shards, "bf16")
        return O.bf16_to_f32(send) if param_dtype == "f32" else send
    impl.ag_pack = rounding_pack
    with pytest.raises(AssertionError):
        C.check_f32_param_roundtrip(impl, 3, [(7, 3), (2, 5)], seed=1)


# ----------------------------------------------------------------- fp16 wires

def run_f16_checks(impl):
    C.check_f16_hex_table(impl)
    C.check_f16_vs_torch(impl)
    C.check_f16_nearest_even(impl)
    for w, dims in SMALL_CASES[:4]:
        C.check_f16_param_roundtrip(impl, w, dims, seed=w)
        C.check_f16_wire(impl, w, dims, w - 1, seed=w)


def test_fp16_variants():
    run_f16_checks(oracle_impl())


def _f16_truncate(x):
    """Round toward zero (what a packed round-toward-zero conversion does)."""
    x = np.asarray(x, np.float32)
    r = x.astype(np.float16)
    back = r.astype(np.float32)
    step = np.nextafter(r, np.float16(0)).astype(np.float16)
    return np.where(np.isfinite(x) & (np.abs(back) > np.abs(x)), step, np.where(np.isinf(r) & np.isfinite(x),
                    np.copysign(np.float16(65504), x).astype(np.float16), r)).astype(np.float16)


def _f16_flush_subnormals(x):
    r = np.asarray(x, np.float32).astype(np.float16)
    return np.where(np.abs(r.astype(np.float32)) < 2.0 ** -14, np.copysign(np.float16(0), r), r).astype(np.float16)


def _f16_via_bf16(x):
    """A cast that rounds to bf16 first (double rounding)."""
    return O.bf16_to_f32(O.bf16_rne(x)).astype(np.float16)


F16_MUTANTS = {
    "fp16 round toward zero": _f16_truncate,
    "fp16 subnormals flushed": _f16_flush_subnormals,
    "fp16 double rounding through bf16": _f16_via_bf16,
}


@pytest.mark.parametrize("name", sorted(F16_MUTANTS))
def test_fp16_pins_catch_mutant(name):
    impl = oracle_impl()
    cast = F16_MUTANTS[name]
    impl.f16_rne = cast

    def pack(plan, rank, shards, param_dtype="bf16"):
        if param_dtype != "f16":
            return O.ag_pack(plan, rank, shards, param_dtype)
        send = np.zeros(plan.chunk, np.float16)
        for p in range(plan.num_params):
            v = O.local_elems(plan, p, rank)
            send[plan.offset[p]:plan.offset[p] + v] = cast(np.asarray(shards[p]).reshape(-1))
        return send
    impl.ag_pack = pack
    with pytest.raises(AssertionError):
        with np.errstate(all="ignore"):
            run_f16_checks(impl)
