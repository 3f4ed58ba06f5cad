"""Checks that pin an auto-wrapping implementation to what the paper and the
mathematics fix (SimpleFSDP section 3.3.2, Algorithm 1, Table 1).

Every check takes ``wrap``, a callable with the signature of
``oracle.auto_wrap.auto_wrap`` returning the buckets as lists of node
indices, and raises AssertionError on a mismatch.  They run against the
oracle (and against the library's host planner); each is independent of the
oracle's code:

* hand-worked tables (tests/golden/auto_wrap_cases.txt);
* closed forms for uniform nodes: forward bucket sizes t**k (alpha = 0) and
  (3**k + 1) / 2 (t = 3, alpha = 1); backward sizes the even-index
  Fibonacci numbers 1, 3, 8, 21, 55, ... (t = 3, reduce-scatter as costly as
  the all-gather);
* special cases: free communication reduces to next-fit bin packing by
  memory; no memory to spare, or no compute to hide behind, gives one node
  per bucket; a free reduce-scatter makes the backward pass equal the
  forward one;
* brute force over every cut of small tables, judged by a timeline
  simulation of the reordered schedule: exactly one cut has every
  multi-node bucket's all-gather hidden behind the step it overlaps and
  within the memory limit, with no bucket able to take the next node; it
  must be the one returned;
* exact scaling: multiplying every time, alpha and beta by a power of two
  changes nothing.
"""

from __future__ import annotations

import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "auto_wrap_cases.txt")


def read_cases(path=GOLDEN):
    """The hand-worked cases: dicts with the model, nodes and expected buckets."""
    cases, cur = [], None
    with open(path) as f:
        for raw in f:
            line = raw.split("#")[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "case":
                cur = dict(name=tok[1], backward=tok[2] == "backward", alpha_ag=float(tok[3]),
                           beta_ag=float(tok[4]), alpha_rs=float(tok[5]), beta_rs=float(tok[6]),
                           mem_max=int(tok[7]), ag=[], rs=[], t=[], m=[])
                cases.append(cur)
            elif tok[0] == "node":
                cur["ag"].append(int(tok[1]))
                cur["rs"].append(int(tok[2]))
                cur["t"].append(float(tok[3]))
                cur["m"].append(int(tok[4]))
            elif tok[0] == "expect":
                rest = line[len("expect"):].strip()
                cur["expect"] = [[int(x) for x in part.split()] for part in rest.split("|")] if rest else []
            else:
                raise ValueError(f"bad line in {path}: {raw!r}")
    return cases


def _call(wrap, c):
    return wrap(c["ag"], c["t"], c["m"], c["alpha_ag"], c["beta_ag"], c["mem_max"], c["backward"],
                c["rs"], c["alpha_rs"], c["beta_rs"])


def check_golden(wrap):
    cases = read_cases()
    assert len(cases) >= 7
    for c in cases:
        got = _call(wrap, c)
        assert got == c["expect"], (c["name"], got, c["expect"])


def _sizes(buckets):
    return [len(b) for b in buckets]


def _contiguous(buckets, n):
    return [i for b in buckets for i in b] == list(range(n))


def check_forward_closed_forms(wrap):
    """Uniform one-word nodes, beta = 1, no memory limit: step k computes for
    t*|B_k|, so the next bucket holds t*|B_k| - alpha nodes."""
    big = 1 << 40
    # alpha = 0, t = 2: 1, 2, 4, 8, 16, 32 and the rest
    n = 70
    got = wrap([1] * n, [2.0] * n, [0] * n, 0.0, 1.0, big)
    assert _contiguous(got, n) and _sizes(got) == [1, 2, 4, 8, 16, 32, 7], _sizes(got)
    # alpha = 1, t = 3: (3**k + 1) / 2 = 1, 2, 5, 14, 41, 122
    n = 1 + 2 + 5 + 14 + 41 + 122 + 3
    got = wrap([1] * n, [3.0] * n, [0] * n, 1.0, 1.0, big)
    assert _contiguous(got, n) and _sizes(got) == [(3 ** k + 1) // 2 for k in range(6)] + [3], _sizes(got)


def check_backward_fibonacci(wrap):
    """Backward pass, uniform one-word nodes, t = 3, alpha = 0 and the
    reduce-scatter costing what the all-gather does: step k hides the
    reduce-scatter of B_{k-1} and the all-gather of B_{k+1}, so
    |B_{k+1}| = 3|B_k| - |B_{k-1}|: the even-index Fibonacci numbers."""
    fib = [1, 1]
    while len(fib) < 16:
        fib.append(fib[-1] + fib[-2])
    want = [fib[2 * k + 1] for k in range(6)]          # 1, 3, 8, 21, 55, 144
    n = sum(want) + 10
    got = wrap([1] * n, [3.0] * n, [0] * n, 0.0, 1.0, 1 << 40, True, [1] * n, 0.0, 1.0)
    assert _contiguous(got, n) and _sizes(got) == want + [10], _sizes(got)
    # an RS twice as costly: |B_{k+1}| = 3|B_k| - 2|B_{k-1}| = 2^(k+1) - 1
    n = 1 + 3 + 7 + 15 + 31 + 5
    got = wrap([1] * n, [3.0] * n, [0] * n, 0.0, 1.0, 1 << 40, True, [2] * n, 0.0, 1.0)
    assert _sizes(got) == [1, 3, 7, 15, 31, 5], _sizes(got)


def _next_fit(sizes, cap):
    """Textbook next-fit bin packing: keep one open bin; an item that does not
    fit closes it and opens a new one."""
    bins, load = [], None
    for i, s in enumerate(sizes):
        if bins and load + s <= cap:
            bins[-1].append(i)
            load += s
        else:
            bins.append([i])
            load = s
    return bins


def check_free_comm_is_next_fit(wrap, seed=0):
    rng = np.random.default_rng(seed)
    for _ in range(50):
        n = int(rng.integers(1, 40))
        mem = [int(x) for x in rng.integers(0, 100, n)]
        cap = int(rng.integers(0, 300))
        t = [float(x) for x in rng.integers(0, 5, n)]
        for backward in (False, True):
            got = wrap([int(x) for x in rng.integers(0, 1000, n)], t, mem, 0.0, 0.0, cap, backward,
                       [int(x) for x in rng.integers(0, 1000, n)], 0.0, 0.0)
            assert got == _next_fit(mem, cap), (got, mem, cap)


def check_singletons(wrap, seed=1):
    rng = np.random.default_rng(seed)
    for _ in range(20):
        n = int(rng.integers(1, 30))
        w = [int(x) for x in rng.integers(1, 50, n)]
        t = [float(x) for x in rng.integers(0, 1000, n)]
        m = [int(x) for x in rng.integers(1, 50, n)]
        # no memory to spare for a second node
        got = wrap(w, t, m, 1.0, 1.0, 0, bool(n % 2), w, 1.0, 1.0)
        assert got == [[i] for i in range(n)]
        # nothing to hide communication behind
        got = wrap(w, [0.0] * n, m, 1e-9, 1.0, 1 << 40)
        assert got == [[i] for i in range(n)]


def check_free_rs_backward_is_forward(wrap, seed=2):
    rng = np.random.default_rng(seed)
    for _ in range(50):
        n = int(rng.integers(1, 30))
        w = [int(x) for x in rng.integers(0, 20, n)]
        t = [float(x) for x in rng.uniform(0, 30, n)]
        m = [int(x) for x in rng.integers(0, 10, n)]
        a, b, cap = float(rng.uniform(0, 3)), float(rng.uniform(0, 2)), int(rng.integers(0, 60))
        fwd = wrap(w, t, m, a, b, cap)
        bwd = wrap(w, t, m, a, b, cap, True, [int(x) for x in rng.integers(0, 20, n)], 0.0, 0.0)
        assert fwd == bwd


def check_power_of_two_scaling(wrap, seed=3):
    rng = np.random.default_rng(seed)
    for _ in range(50):
        n = int(rng.integers(1, 30))
        w = [int(x) for x in rng.integers(0, 1 << 20, n)]
        r = [int(x) for x in rng.integers(0, 1 << 20, n)]
        t = [float(x) for x in rng.uniform(0, 1e-3, n)]
        m = [int(x) for x in rng.integers(0, 1 << 30, n)]
        a, b = float(rng.uniform(0, 1e-5)), float(rng.uniform(0, 1e-9))
        ar, br = float(rng.uniform(0, 1e-5)), float(rng.uniform(0, 2e-9))
        cap = int(rng.integers(0, 1 << 32))
        for backward in (False, True):
            base = wrap(w, t, m, a, b, cap, backward, r, ar, br)
            for e in (-7, 11):
                s = 2.0 ** e
                got = wrap(w, [x * s for x in t], m, a * s, b * s, cap, backward, r, ar * s, br * s)
                assert got == base


# ---------------------------------------------------------------- brute force

def simulate(buckets, ag, rs, t, m, alpha_ag, beta_ag, alpha_rs, beta_rs, backward):
    """Timeline of one pass under the reordered schedule: one compute stream,
    one in-order communication stream.  The all-gather of B_0 is issued at
    time 0; at the start of step k the all-gather of B_{k+1} is issued, and
    (backward) the reduce-scatter of B_{k-1} when step k-1 ends; step k starts
    once its own all-gather is done.  Returns each step's stall (the time the
    compute stream waits for that step's all-gather) and each bucket's memory."""
    def t_ag(b):
        return alpha_ag + beta_ag * sum(ag[i] for i in b)

    def t_rs(b):
        return alpha_rs + beta_rs * sum(rs[i] for i in b)

    K = len(buckets)
    comm_free = 0.0
    ag_done = [0.0] * K
    if K:
        ag_done[0] = comm_free = t_ag(buckets[0])
    end_prev = 0.0
    stalls = []
    for k in range(K):
        start = max(end_prev, ag_done[k])
        stalls.append(start - end_prev)
        if backward and k >= 1:
            comm_free = max(end_prev, comm_free) + t_rs(buckets[k - 1])
        if k + 1 < K:
            ag_done[k + 1] = comm_free = max(start, comm_free) + t_ag(buckets[k + 1])
        end_prev = start + sum(t[i] for i in buckets[k])
    mems = [sum(m[i] for i in b) for b in buckets]
    return stalls, mems


def _cuts(n):
    """Every way to cut 0..n-1 into consecutive non-empty buckets."""
    for mask in range(1 << max(n - 1, 0)):
        buckets, cur = [], [0]
        for i in range(1, n):
            if mask >> (i - 1) & 1:
                buckets.append(cur)
                cur = [i]
            else:
                cur.append(i)
        yield buckets + [cur] if n else []


def _legal(bk, stall, mem, mem_max):
    return len(bk) == 1 or (stall == 0 and mem <= mem_max)


def _is_auto_wrap(buckets, args, mem_max):
    stalls, mems = simulate(buckets, *args)
    if not all(_legal(b, s, mm, mem_max) for b, s, mm in zip(buckets, stalls, mems)):
        return False
    for k in range(len(buckets) - 1):
        # bucket k must not be able to take the next node as well
        moved = [list(b) for b in buckets]
        moved[k].append(moved[k + 1].pop(0))
        moved = [b for b in moved if b]
        s2, m2 = simulate(moved, *args)
        if _legal(moved[k], s2[k], m2[k], mem_max):
            return False
    return True


def check_bruteforce(wrap, n_cases=150, seed=4, max_n=8):
    """Small integer-valued tables (every sum is exact, ties are frequent)."""
    rng = np.random.default_rng(seed)
    for case in range(n_cases):
        n = int(rng.integers(0, max_n + 1))
        ag = [int(x) for x in rng.integers(0, 6, n)]
        rs = [int(x) for x in rng.integers(0, 6, n)]
        t = [float(x) for x in rng.integers(0, 13, n)]
        m = [int(x) for x in rng.integers(0, 6, n)]
        mem_max = int(rng.integers(0, 13))
        a, b, ar, br = (float(x) for x in rng.integers(0, 3, 4))
        backward = bool(case % 2)
        args = (ag, rs, t, m, a, b, ar, br, backward)
        found = [c for c in _cuts(n) if _is_auto_wrap(c, args, mem_max)]
        assert len(found) == 1, (case, found)
        got = wrap(ag, t, m, a, b, mem_max, backward, rs, ar, br)
        assert got == found[0], (case, got, found[0], args, mem_max)


def run_all(wrap, quick=False):
    check_golden(wrap)
    check_forward_closed_forms(wrap)
    check_backward_fibonacci(wrap)
    check_free_comm_is_next_fit(wrap)
    check_singletons(wrap)
    check_free_rs_backward_is_forward(wrap)
    check_power_of_two_scaling(wrap)
    check_bruteforce(wrap, n_cases=60 if quick else 300)

