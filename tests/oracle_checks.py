"""Pins for the CPU oracle, written as checks over an implementation namespace.

Each check takes ``impl`` (a namespace with ``make_plan``, ``local_rows``,
``bf16_rne``, ``ag_pack``, ``ag_unpack``, ``rs_pack``, ``rs_reduce``) and
raises AssertionError on a mismatch.  ``test_oracle_pins`` runs them against
the real oracle (all must pass) and against deliberately broken copies of it
(each must be caught by at least one check), so a pin that cannot fail is
noticed.

None of these checks retypes the oracle's formulas: they compare against
hand-worked tables, torch library routines (``torch.chunk``, the CPU bf16
cast), per-element brute force written in a different style (Python scalars,
float64 arithmetic rounded once to fp32), closed forms and invariants.
"""

from __future__ import annotations

import math
import os

import numpy as np
import torch

from synth import random_bits32, exact_grad_bits

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ---------------------------------------------------------------- helpers

def read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append(line.split())
    return rows


def f32_from_bits(u):
    return np.asarray(u, dtype=np.uint32).view(np.float32)


def torch_bf16_bits(x_f32: np.ndarray) -> np.ndarray:
    """bf16 bits via torch's CPU cast (a library routine)."""
    t = torch.from_numpy(np.ascontiguousarray(x_f32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_float(b: int) -> float:
    """Value of a bf16 bit pattern as a Python float, from its fields."""
    sign = -1.0 if (b >> 15) & 1 else 1.0
    e = (b >> 7) & 0xFF
    m = b & 0x7F
    if e == 0xFF:
        return sign * math.inf if m == 0 else math.nan
    if e == 0:
        return sign * m * 2.0 ** (-133)          # subnormal: m * 2^-7 * 2^-126
    return sign * (1.0 + m / 128.0) * 2.0 ** (e - 127)


def torch_chunk_rows(n: int, w: int) -> list[int]:
    """Rows per rank of a dim-0 ``torch.chunk`` split (what DTensor Shard(0) uses)."""
    parts = torch.chunk(torch.empty(n, 1), w, dim=0) if n > 0 else ()
    rows = [p.shape[0] for p in parts]
    return rows + [0] * (w - len(rows))


def round_f32(x: float) -> float:
    """Round a Python float (binary64) to the nearest binary32, ties to even."""
    return float(np.float32(x))


# ---------------------------------------------------------------- bf16 cast

def check_bf16_hex_table(impl):
    for inp, out, *_ in read_table("bf16_rne_cases.txt"):
        got = int(impl.bf16_rne(f32_from_bits([int(inp, 16)]))[0])
        assert got == int(out, 16), f"bf16({inp}) = {got:#06x}, table says {out}"


def check_bf16_vs_torch(impl, n=1 << 18):
    u = random_bits32([7, 1], n)
    x = f32_from_bits(u)
    finite = ~np.isnan(x)
    ours = impl.bf16_rne(x)
    ref = torch_bf16_bits(x)
    assert np.array_equal(ours[finite], ref[finite])
    assert np.all(np.isnan(f32_from_bits(ours[~finite].astype(np.uint32) << 16)))


def check_bf16_nearest_even(impl, n=4000):
    """Brute force from the definition: the nearer of the two bf16 neighbours."""
    u = random_bits32([7, 2], n)
    x = f32_from_bits(u)
    got = impl.bf16_rne(x)
    for k in range(n):
        xv = float(x[k])
        if math.isnan(xv) or math.isinf(xv):
            continue
        lo = int(u[k]) >> 16                      # truncation toward zero
        hi = lo + 1                               # next bf16 away from zero
        vlo, vhi = bf16_bits_to_float(lo), bf16_bits_to_float(hi)
        dlo, dhi = abs(xv - vlo), abs(vhi - xv) if not math.isinf(vhi) else None
        if dhi is None:
            # above the largest finite bf16: overflow threshold is half an ulp
            limit = bf16_bits_to_float(lo) + 2.0 ** (127 - 8)
            want = hi if abs(xv) >= limit and (abs(xv) > limit or (lo & 1)) else lo
        elif dlo < dhi:
            want = lo
        elif dhi < dlo:
            want = hi
        else:
            want = lo if (lo & 1) == 0 else hi
        assert int(got[k]) == want, f"x={u[k]:#010x} got {int(got[k]):#06x} want {want:#06x}"


def check_bf16_nan(impl):
    for u in (0x7FC00000, 0xFFC00000, 0x7F800001, 0xFF800001, 0x7FFFFFFF):
        b = int(impl.bf16_rne(f32_from_bits([u]))[0])
        assert (b & 0x7F80) == 0x7F80 and (b & 0x7F) != 0, f"NaN {u:#x} -> {b:#x}"
        assert (b >> 15) == (u >> 31)


# ---------------------------------------------------------------- plan

def check_plan_toy_table(impl):
    rows = read_table("plan_toy_w4.txt")
    dims = [(int(r[1]), int(r[2])) for r in rows]
    plan = impl.make_plan(4, dims, 8)
    for p, r in enumerate(rows):
        assert plan.rows_per_rank[p] == int(r[3])
        assert plan.offset[p] == int(r[4])
        assert plan.seg[p] == int(r[5])
    assert plan.chunk == 197760
    assert 4 * plan.chunk == sum(n * k for n, k in dims)


def check_plan_sharding_matches_torch_chunk(impl, cases):
    for w, dims in cases:
        plan = impl.make_plan(w, dims, 8)
        for p, (n, _) in enumerate(dims):
            want = torch_chunk_rows(n, w)
            got = [impl.local_rows(plan, p, r) for r in range(w)]
            assert got == want, (w, n, got, want)


def check_plan_invariants(impl, cases):
    for w, dims in cases:
        for a in (1, 2, 8, 16):
            plan = impl.make_plan(w, dims, a)
            end = 0
            for p, (n, k) in enumerate(dims):
                o = plan.offset[p]
                assert o % a == 0                      # aligned start
                assert end <= o < end + a              # after the previous one, gap < a
                # the segment holds exactly one rank's rows of the padded tensor
                assert plan.seg[p] == plan.rows_per_rank[p] * k
                assert sum(impl.local_rows(plan, p, r) for r in range(w)) == n
                end = o + plan.seg[p]
            assert plan.chunk % a == 0 and end <= plan.chunk < end + a
            assert w * plan.chunk >= sum(n * k for n, k in dims)
            if a == 1:
                # dense flatten-and-concatenate: no gaps at all
                assert plan.chunk == sum(plan.seg)


def check_plan_even_workloads(impl, workloads):
    """Blocks whose every dim 0 divides by W and whose segments are 8-aligned:
    the bucket holds no padding, so W * S equals the element count exactly."""
    for wl in workloads:
        plan = impl.make_plan(wl.world_size, wl.dims, 8)
        assert wl.world_size * plan.chunk == wl.total_elems, wl.name


# ---------------------------------------------------------------- brute force pack/unpack

def _find_param(plan, k):
    for p in range(plan.num_params):
        if plan.offset[p] <= k < plan.offset[p] + plan.seg[p]:
            return p
    return None


def check_ag_pack_bruteforce(impl, w, dims, rank, seed, align=8):
    plan = impl.make_plan(w, dims, align)
    full = []
    shards = []
    for p, (n, k) in enumerate(dims):
        x = f32_from_bits(random_bits32([seed, p], n * k)).reshape(n, k)
        full.append(x)
        shards.append(torch.chunk(torch.from_numpy(x), w, dim=0))
    local = []
    for p, (n, k) in enumerate(dims):
        parts = shards[p]
        local.append(parts[rank].numpy() if rank < len(parts) else np.zeros((0, k), np.float32))
    got = impl.ag_pack(plan, rank, local)
    assert got.shape == (plan.chunk,)
    for kk in range(plan.chunk):
        p = _find_param(plan, kk)
        if p is None:
            assert got[kk] == 0, f"gap/tail {kk} not zero"
            continue
        n, k = dims[p]
        e = kk - plan.offset[p]
        q, col = divmod(e, k)
        row = rank * plan.rows_per_rank[p] + q
        if q < plan.rows_per_rank[p] and row < n:
            want = torch_bf16_bits(full[p][row:row + 1, col])[0]
            if math.isnan(float(full[p][row, col])):
                assert (int(got[kk]) & 0x7F80) == 0x7F80 and (int(got[kk]) & 0x7F)
                continue
            assert got[kk] == want, (p, row, col)
        else:
            assert got[kk] == 0, f"pad row {row} of param {p} not zero"


def check_ag_unpack_bruteforce(impl, w, dims, seed, align=8):
    plan = impl.make_plan(w, dims, align)
    S = plan.chunk
    g = (random_bits32([seed, 99], w * S) & 0xFFFF).astype(np.uint16)
    out = impl.ag_unpack(plan, g)
    for p, (n, k) in enumerate(dims):
        assert out[p].shape == (n, k)
        c = plan.rows_per_rank[p]
        for row in range(n):
            i, q = divmod(row, c)
            for col in range(k):
                assert out[p][row, col] == g[i * S + plan.offset[p] + q * k + col]


def check_rs_pack_bruteforce(impl, w, dims, seed, align=8):
    plan = impl.make_plan(w, dims, align)
    S = plan.chunk
    grads = [(random_bits32([seed, p, 5], n * k) & 0xFFFF).astype(np.uint16).reshape(n, k)
             for p, (n, k) in enumerate(dims)]
    send = impl.rs_pack(plan, grads)
    assert send.shape == (w * S,)
    for j in range(w):
        for kk in range(S):
            p = _find_param(plan, kk)
            v = int(send[j * S + kk])
            if p is None:
                assert v == 0
                continue
            n, k = dims[p]
            q, col = divmod(kk - plan.offset[p], k)
            row = j * plan.rows_per_rank[p] + q
            assert v == (int(grads[p][row, col]) if row < n else 0), (j, kk, p, row, col)


def check_roundtrip_library(impl, w, dims, seed, align=8):
    """unpack(all_gather(pack_r(chunk_r(X)))) == X cast by torch, for every rank layout."""
    plan = impl.make_plan(w, dims, align)
    xs = [np.asarray(np.random.default_rng([seed, p]).standard_normal((n, k)), np.float32)
          for p, (n, k) in enumerate(dims)]
    chunks = []
    for r in range(w):
        local = []
        for p, (n, k) in enumerate(dims):
            parts = torch.chunk(torch.from_numpy(xs[p]), w, dim=0) if n else ()
            local.append(parts[r].numpy() if r < len(parts) else np.zeros((0, k), np.float32))
        chunks.append(impl.ag_pack(plan, r, local))
    gathered = np.concatenate(chunks)
    out = impl.ag_unpack(plan, gathered)
    for p in range(len(dims)):
        assert np.array_equal(out[p], torch_bf16_bits(xs[p]).reshape(xs[p].shape)), p


def check_rs_pack_equals_ag_layout(impl, w, dims, seed, align=8):
    """For bf16-representable G, rs_pack(G) == concat_r ag_pack_r(chunk_r(G)):
    both buffers use the same per-rank [W][S] layout."""
    plan = impl.make_plan(w, dims, align)
    grads = [exact_grad_bits([seed, p], (n, k)) for p, (n, k) in enumerate(dims)]
    send = impl.rs_pack(plan, grads)
    parts = []
    for r in range(w):
        local = []
        for p, (n, k) in enumerate(dims):
            gf = (grads[p].astype(np.uint32) << 16).view(np.float32)
            ch = torch.chunk(torch.from_numpy(gf), w, dim=0) if n else ()
            local.append(ch[r].numpy() if r < len(ch) else np.zeros((0, k), np.float32))
        parts.append(impl.ag_pack(plan, r, local))
    assert np.array_equal(send, np.concatenate(parts))


# ---------------------------------------------------------------- reduction

def _exchange(send_bufs, rank, S):
    return np.concatenate([b[rank * S:(rank + 1) * S] for b in send_bufs])


def check_rs_reduce_bruteforce(impl, w, dims, rank, seed, align=8, exact=False):
    """Per element: binary64 arithmetic rounded to binary32 after every step.

    Rounding a binary64 sum or quotient of binary32 operands to binary32 gives
    the correctly rounded binary32 result (53 >= 2*24 + 2), so this loop is an
    independent route to fl32(fl32(x0 + x1) + ...) / W.  Padding in the
    receive buffer is never read, so the whole buffer is filled with data.
    """
    plan = impl.make_plan(w, dims, align)
    S = plan.chunk
    if exact:
        recv = exact_grad_bits([seed, 3], w * S)
    else:
        # magnitudes spread over 2^-24..2^24 so that fp32 sums round and the
        # summation order shows in the result bits
        rng = np.random.default_rng([seed, 3])
        g = rng.standard_normal(w * S) * np.exp2(rng.integers(-24, 25, w * S))
        recv = torch_bf16_bits(g.astype(np.float32))
    out = impl.rs_reduce(plan, rank, recv)
    for p, (n, k) in enumerate(dims):
        nr = impl.local_rows(plan, p, rank)
        assert out[p].shape == (nr, k)
        flat = out[p].reshape(-1)
        for e in range(nr * k):
            a = bf16_bits_to_float(int(recv[plan.offset[p] + e]))
            for i in range(1, w):
                a = round_f32(a + bf16_bits_to_float(int(recv[i * S + plan.offset[p] + e])))
            a = round_f32(a / w)
            assert float(flat[e]) == a or (math.isnan(a) and math.isnan(float(flat[e]))), (p, e)
    return recv, out


def check_rs_reduce_closed_forms(impl):
    # W = 1: the identity (x0 / 1)
    plan = impl.make_plan(1, [(5, 3)], 8)
    recv = torch_bf16_bits(np.linspace(-3, 3, plan.chunk).astype(np.float32))
    out = impl.rs_reduce(plan, 0, recv)[0].reshape(-1)
    want = (recv[:15].astype(np.uint32) << 16).view(np.float32)
    assert np.array_equal(out, want)
    # W = 2^k: the quotient is an exact power-of-two scaling of the fp32 sum
    for w in (2, 4, 8, 16):
        plan = impl.make_plan(w, [(w * 3, 5)], 8)
        S = plan.chunk
        recv = exact_grad_bits([11, w], w * S)
        out = impl.rs_reduce(plan, 1, recv)[0].reshape(-1)
        v = out.size
        for e in range(v):
            s = sum(bf16_bits_to_float(int(recv[i * S + plan.offset[0] + e])) for i in range(w))
            assert float(out[e]) == s * 2.0 ** -int(math.log2(w)), (w, e)
    # signed zeros: all -0 stays -0 (the sum starts from x0, not from +0)
    for w in (1, 3):
        plan = impl.make_plan(w, [(w, 2)], 8)
        recv = np.full(w * plan.chunk, 0x8000, np.uint16)
        out = impl.rs_reduce(plan, 0, recv)[0].reshape(-1)
        assert np.all(np.signbit(out)) and np.all(out == 0)
    # inf + (-inf) = NaN, inf + finite = inf
    plan = impl.make_plan(2, [(2, 2)], 8)
    S = plan.chunk
    recv = np.zeros(2 * S, np.uint16)
    recv[0], recv[S] = 0x7F80, 0xFF80
    recv[1], recv[S + 1] = 0x7F80, 0x3F80
    out = impl.rs_reduce(plan, 0, recv)[0].reshape(-1)
    assert math.isnan(out[0]) and out[1] == np.inf
    # subnormals survive: 2 * tiny / 2 == tiny
    recv = np.zeros(2 * S, np.uint16)
    recv[0] = recv[S] = 0x0001                    # smallest bf16 subnormal
    out = impl.rs_reduce(plan, 0, recv)[0].reshape(-1)
    assert out[0] == np.float32(2.0 ** -133)


def check_rs_reduce_not_reciprocal(impl):
    """W = 48: a correctly rounded x/48 differs from x*(1/48) for many x; the
    brute force above fixes which one is meant; here the reduction must give
    the quotient on inputs where the two disagree."""
    w = 48
    plan = impl.make_plan(w, [(w * 4, 8)], 8)
    S = plan.chunk
    g = np.random.default_rng(48).standard_normal(w * S).astype(np.float32)
    recv = torch_bf16_bits(g)
    out = impl.rs_reduce(plan, 0, recv)[0].reshape(-1)
    v = out.size
    sums = []
    for e in range(v):
        a = bf16_bits_to_float(int(recv[e]))
        for i in range(1, w):
            a = round_f32(a + bf16_bits_to_float(int(recv[i * S + e])))
        sums.append(a)
    quo = np.array([round_f32(s / w) for s in sums], np.float32)
    rec = np.array([round_f32(s * float(np.float32(1.0 / 48))) for s in sums], np.float32)
    assert np.count_nonzero(quo != rec) > 0, "test inputs do not separate x/48 from x*(1/48)"
    assert np.array_equal(out, quo)


def check_ag_then_rs_replicated(impl, w, dims, seed, align=8):
    """The gathered bf16 parameter fed back as every rank's gradient returns the
    rank's bf16 shard exactly: W copies of a bf16 value sum exactly in fp32
    (8-bit significand, W <= 2^16) and the correctly rounded (W*x)/W is x."""
    plan = impl.make_plan(w, dims, align)
    S = plan.chunk
    xs = [np.random.default_rng([seed, p]).standard_normal((n, k)).astype(np.float32)
          for p, (n, k) in enumerate(dims)]
    chunks = []
    for r in range(w):
        local = []
        for p, (n, k) in enumerate(dims):
            ch = torch.chunk(torch.from_numpy(xs[p]), w, dim=0) if n else ()
            local.append(ch[r].numpy() if r < len(ch) else np.zeros((0, k), np.float32))
        chunks.append(impl.ag_pack(plan, r, local))
    full = impl.ag_unpack(plan, np.concatenate(chunks))
    send = impl.rs_pack(plan, full)            # every rank holds the same gradient
    for j in sorted({0, w // 2, w - 1}):
        recv = _exchange([send] * w, j, S)
        out = impl.rs_reduce(plan, j, recv)
        for p, (n, k) in enumerate(dims):
            ch = torch.chunk(torch.from_numpy(xs[p]), w, dim=0) if n else ()
            want = ch[j].numpy() if j < len(ch) else np.zeros((0, k), np.float32)
            want = (torch_bf16_bits(want).astype(np.uint32) << 16).view(np.float32).reshape(want.shape)
            assert np.array_equal(out[p], want), (w, j, p)


def check_rs_exact_mean_bound(impl, w, seed):
    """Sanity bound of a sequential fp32 sum against the exact mean."""
    plan = impl.make_plan(w, [(w * 16, 32)], 8)
    S = plan.chunk
    g = np.random.default_rng([seed, w]).standard_normal(w * S).astype(np.float32)
    recv = torch_bf16_bits(g)
    out = impl.rs_reduce(plan, 0, recv)[0].reshape(-1).astype(np.float64)
    v = out.size
    x = (recv.astype(np.uint32) << 16).view(np.float32).astype(np.float64).reshape(w, S)[:, :v]
    mean = x.sum(axis=0) / w
    bound = (w - 1) * 2.0 ** -24 * np.abs(x).sum(axis=0) / w + np.abs(mean) * 2.0 ** -24 + 1e-45
    assert np.all(np.abs(out - mean) <= bound)


# ---------------------------------------------------------------- fp32 variants

def check_f32_param_roundtrip(impl, w, dims, seed, align=8):
    """Without mixed precision (param_dtype fp32) the all-gather reproduces the
    fp32 parameter bit for bit, NaN payloads included."""
    plan = impl.make_plan(w, dims, align)
    xs = [f32_from_bits(random_bits32([seed, p, 11], n * k)).reshape(n, k) for p, (n, k) in enumerate(dims)]
    chunks = []
    for r in range(w):
        local = []
        for p, (n, k) in enumerate(dims):
            parts = torch.chunk(torch.from_numpy(xs[p]), w, dim=0) if n else ()
            local.append(parts[r].numpy() if r < len(parts) else np.zeros((0, k), np.float32))
        send = impl.ag_pack(plan, r, local, param_dtype="f32")
        assert send.dtype == np.float32 and send.shape == (plan.chunk,)
        # padding is +0.0 in fp32 too
        mask = np.ones(plan.chunk, bool)
        for p in range(len(dims)):
            v = impl.local_rows(plan, p, r) * dims[p][1]
            mask[plan.offset[p]:plan.offset[p] + v] = False
        assert np.all(send.view(np.uint32)[mask] == 0)
        chunks.append(send)
    out = impl.ag_unpack(plan, np.concatenate(chunks))
    for p in range(len(dims)):
        assert out[p].dtype == np.float32
        assert np.array_equal(out[p].view(np.uint32), xs[p].view(np.uint32)), p


def check_f32_wire_same_bits(impl, w, dims, seed, align=8):
    """An fp32 reduce-scatter wire (gradients cast to reduce_dtype before the
    exchange) gives the same result bits as the bf16 wire: widening is exact."""
    plan = impl.make_plan(w, dims, align)
    S = plan.chunk
    rng = np.random.default_rng([seed, 12])
    grads = []
    for i in range(w):
        gi = []
        for n, k in dims:
            f = rng.standard_normal((n, k)) * np.exp2(rng.integers(-24, 25, (n, k)))
            gi.append((f.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16))
        grads.append(gi)
    s16 = [impl.rs_pack(plan, g) for g in grads]
    s32 = [impl.rs_pack(plan, g, reduce_dtype="f32") for g in grads]
    for a, b in zip(s16, s32):
        assert b.dtype == np.float32
        assert np.array_equal((a.astype(np.uint32) << 16), b.view(np.uint32))
    for j in sorted({0, w // 2, w - 1}):
        r16 = impl.rs_reduce(plan, j, _exchange(s16, j, S))
        r32 = impl.rs_reduce(plan, j, _exchange(s32, j, S))
        for p in range(len(dims)):
            assert np.array_equal(r16[p].view(np.uint32), r32[p].view(np.uint32)), (j, p)


def check_rs_reduce_bruteforce_f32(impl, w, dims, rank, seed, align=8):
    """fp32 inputs (full 24-bit significands, wide exponents): the same
    binary64-rounded-per-step brute force as for bf16 inputs."""
    plan = impl.make_plan(w, dims, align)
    S = plan.chunk
    rng = np.random.default_rng([seed, 13])
    recv = (rng.standard_normal(w * S) * np.exp2(rng.integers(-30, 31, w * S))).astype(np.float32)
    out = impl.rs_reduce(plan, rank, recv)
    for p, (n, k) in enumerate(dims):
        nr = impl.local_rows(plan, p, rank)
        flat = out[p].reshape(-1)
        assert flat.size == nr * k
        for e in range(nr * k):
            a = float(recv[plan.offset[p] + e])
            for i in range(1, w):
                a = round_f32(a + float(recv[i * S + plan.offset[p] + e]))
            assert float(flat[e]) == round_f32(a / w), (p, e)


# ---------------------------------------------------------------- fp16 variants

def f16_bits_to_float(b: int) -> float:
    """Decode a binary16 bit pattern from its fields (no numpy float16)."""
    sign = -1.0 if b >> 15 else 1.0
    e = (b >> 10) & 0x1F
    m = b & 0x3FF
    if e == 0x1F:
        return sign * math.inf if m == 0 else math.nan
    if e == 0:
        return sign * m * 2.0 ** -24
    return sign * (1.0 + m / 1024.0) * 2.0 ** (e - 15)


def _f16_bits(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float16).view(np.uint16)


def check_f16_hex_table(impl):
    for inp, out, *_ in read_table("f16_rne_cases.txt"):
        got = int(_f16_bits(impl.f16_rne(f32_from_bits([int(inp, 16)])))[0])
        assert got == int(out, 16), f"f16({inp}) = {got:#06x}, table says {out}"


def check_f16_vs_torch(impl, n=1 << 16):
    u = random_bits32([7, 21], n)
    x = f32_from_bits(u)
    ours = _f16_bits(impl.f16_rne(x))
    ref = torch.from_numpy(x.copy()).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(x)
    assert np.array_equal(ours[~nan], ref[~nan])
    o = ours[nan]
    assert np.all(((o & 0x7C00) == 0x7C00) & ((o & 0x3FF) != 0))


def check_f16_nearest_even(impl, n=400):
    """Brute force from the definition: the nearest of all finite binary16
    values (decoded from their fields), ties to an even significand, and
    infinity at or beyond the largest finite value plus half an ulp."""
    codes = np.arange(0, 0x7C00, dtype=np.int64)                 # finite, non-negative
    vals = np.array([f16_bits_to_float(int(c)) for c in codes])
    rng = np.random.default_rng([7, 22])
    mant = rng.standard_normal(n) * np.exp2(rng.integers(-27, 18, n))
    x = mant.astype(np.float32)
    got = _f16_bits(impl.f16_rne(x))
    limit = 65504.0 + 16.0                                       # half an ulp above the top
    for k in range(n):
        xv = float(x[k])
        a = abs(xv)
        if a >= limit:
            want = 0x7C00
        else:
            d = np.abs(vals - a)
            best = np.flatnonzero(d == d.min())
            want = int(codes[best[0]]) if best.size == 1 else int(codes[best[np.argmax(codes[best] % 2 == 0)]])
        if xv < 0 or (xv == 0 and math.copysign(1.0, xv) < 0):
            want |= 0x8000
        assert int(got[k]) == want, f"x={xv!r} got {int(got[k]):#06x} want {want:#06x}"


def check_f16_param_roundtrip(impl, w, dims, seed, align=8):
    """param_dtype fp16: the gathered, unpacked parameters equal torch's fp16
    cast of the full fp32 parameters; padding is +0."""
    plan = impl.make_plan(w, dims, align)
    xs = [np.asarray(np.random.default_rng([seed, p, 23]).standard_normal((n, k))
                     * np.exp2(np.random.default_rng([seed, p, 24]).integers(-26, 18, (n, k))), np.float32)
          for p, (n, k) in enumerate(dims)]
    chunks = []
    for r in range(w):
        local = []
        for p, (n, k) in enumerate(dims):
            parts = torch.chunk(torch.from_numpy(xs[p]), w, dim=0) if n else ()
            local.append(parts[r].numpy() if r < len(parts) else np.zeros((0, k), np.float32))
        send = impl.ag_pack(plan, r, local, param_dtype="f16")
        assert send.dtype == np.float16 and send.shape == (plan.chunk,)
        mask = np.ones(plan.chunk, bool)
        for p in range(len(dims)):
            v = impl.local_rows(plan, p, r) * dims[p][1]
            mask[plan.offset[p]:plan.offset[p] + v] = False
        assert np.all(_f16_bits(send)[mask] == 0)
        chunks.append(send)
    out = impl.ag_unpack(plan, np.concatenate(chunks))
    for p in range(len(dims)):
        want = torch.from_numpy(xs[p]).to(torch.float16).view(torch.int16).numpy().view(np.uint16)
        assert out[p].dtype == np.float16
        assert np.array_equal(_f16_bits(out[p]), want), p


def check_f16_wire(impl, w, dims, rank, seed, align=8):
    """fp16 gradients: an fp16 wire and an fp32 wire give the same bits
    (widening is exact), and each output equals the binary64-rounded-per-step
    brute force over the decoded fp16 inputs."""
    plan = impl.make_plan(w, dims, align)
    S = plan.chunk
    rng = np.random.default_rng([seed, 25])
    grads = []
    for i in range(w):
        gi = []
        for n, k in dims:
            bits = (rng.integers(0, 0x7C00, (n, k)) | (rng.integers(0, 2, (n, k)) << 15)).astype(np.uint16)
            gi.append(bits.view(np.float16))
        grads.append(gi)
    s16 = [impl.rs_pack(plan, g, reduce_dtype="f16") for g in grads]
    s32 = [impl.rs_pack(plan, g, reduce_dtype="f32") for g in grads]
    for a, b in zip(s16, s32):
        assert a.dtype == np.float16 and b.dtype == np.float32
        dec = np.array([f16_bits_to_float(int(v)) for v in _f16_bits(a)[:4096]])
        assert np.array_equal(dec, b[:4096].astype(np.float64))
    recv16 = _exchange(s16, rank, S)
    r16 = impl.rs_reduce(plan, rank, recv16)
    r32 = impl.rs_reduce(plan, rank, _exchange(s32, rank, S))
    bits = _f16_bits(recv16)
    for p, (n, k) in enumerate(dims):
        assert np.array_equal(r16[p].view(np.uint32), r32[p].view(np.uint32)), p
        nr = impl.local_rows(plan, p, rank)
        flat = r16[p].reshape(-1)
        for e in range(nr * k):
            a_ = f16_bits_to_float(int(bits[plan.offset[p] + e]))
            for i in range(1, w):
                a_ = round_f32(a_ + f16_bits_to_float(int(bits[i * S + plan.offset[p] + e])))
            assert float(flat[e]) == round_f32(a_ / w), (p, e)
