"""The library's auto-wrapping planner (``fsdp_auto_wrap``, host code, no GPU)
against the oracle and against the same pins the oracle passes."""

from __future__ import annotations

import ctypes
import time

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import auto_wrap_checks as C
from oracle.auto_wrap import auto_wrap as oracle_wrap

native = pytest.importorskip("paper_2411_00284_amd._native")
LIB = native.load()

from paper_2411_00284_amd import FsdpError, auto_wrap  # noqa: E402

INVALID, OVERFLOW = 1, 3


def test_library_passes_every_pin():
    C.run_all(auto_wrap)


# Times drawn from values whose sums round (0.1 + 0.2 != 0.3), so a different
# summation order or a fused multiply-add would show up as a different cut.
TIMES = [0.0, 0.1, 0.2, 0.3, 0.7, 1e-3, 3.0, 1.0 / 3.0]
COEFS = [0.0, 0.1, 0.2, 0.3, 1e-3, 1.0 / 3.0]


@settings(max_examples=400, deadline=None)
@given(st.data())
def test_library_equals_oracle(data):
    n = data.draw(st.integers(0, 40))
    ag = data.draw(st.lists(st.integers(0, 9), min_size=n, max_size=n))
    rs = data.draw(st.lists(st.integers(0, 9), min_size=n, max_size=n))
    t = data.draw(st.lists(st.sampled_from(TIMES) | st.floats(0, 10), min_size=n, max_size=n))
    m = data.draw(st.lists(st.integers(0, 9), min_size=n, max_size=n))
    a, b, ar, br = (data.draw(st.sampled_from(COEFS) | st.floats(0, 2)) for _ in range(4))
    mem_max = data.draw(st.integers(0, 40))
    backward = data.draw(st.booleans())
    want = oracle_wrap(ag, t, m, a, b, mem_max, backward, rs, ar, br)
    got = auto_wrap(ag, t, m, a, b, mem_max, backward, rs, ar, br)
    assert got == want


def test_library_equals_oracle_llama_like():
    """A Llama-like pass: 80 blocks of 9 tensors (attention, FFN, norms), words
    from their padded all-gathers at W = 64, compute times and activation
    memories of a plausible scale, both directions."""
    rng = np.random.default_rng(7)
    dims = [(8192, 8192), (1024, 8192), (1024, 8192), (8192, 8192), (28672, 8192), (28672, 8192),
            (8192, 28672), (8192, 1), (8192, 1)]
    W = 64
    ag, t, m = [], [], []
    for _ in range(80):
        for n, k in dims:
            ag.append(W * (-(-n // W)) * k)
            t.append(float(n * k) * 2 * 8192 / 1e15 * rng.uniform(0.9, 1.1))   # seconds of compute
            m.append(int(2 * n * k + rng.integers(0, 1 << 24)))
    rs = list(ag)
    for alpha, beta, mem_max in ((20e-6, 2 / 50e9, 8 << 30), (5e-6, 2 / 150e9, 2 << 30), (0.0, 0.0, 1 << 40)):
        for backward in (False, True):
            want = oracle_wrap(ag, t, m, alpha, beta, mem_max, backward, rs, alpha * 1.5, beta * 2)
            got = auto_wrap(ag, t, m, alpha, beta, mem_max, backward, rs, alpha * 1.5, beta * 2)
            assert got == want
            assert 1 <= len(got) <= len(ag)


def test_large_pass_is_linear_time():
    n = 1_000_000
    rng = np.random.default_rng(3)
    ag = rng.integers(1, 1000, n).tolist()
    t = rng.uniform(0, 1e-3, n).tolist()
    m = rng.integers(0, 1000, n).tolist()
    t0 = time.perf_counter()
    got = auto_wrap(ag, t, m, 1e-4, 1e-7, 50_000, True, ag, 1e-4, 2e-7)
    dt = time.perf_counter() - t0
    assert sum(len(b) for b in got) == n
    assert dt < 10.0


# ---------------------------------------------------------------- error paths

def _raw(n, backward=0, ag=None, rs=None, t=None, m=None, a=(0.0, 0.0, 0.0, 0.0), mem_max=10,
         out=True, nb=True):
    A64 = ctypes.c_int64 * max(n, 1)
    D = ctypes.c_double * max(n, 1)
    ag = A64(*(ag if ag is not None else [1] * n))
    rs = None if rs == "null" else A64(*(rs if rs is not None else [1] * n))
    t = D(*(t if t is not None else [1.0] * n))
    m = A64(*(m if m is not None else [1] * n))
    bucket_of = (ctypes.c_int32 * max(n, 1))(*([-7] * max(n, 1)))
    nbv = ctypes.c_int32(-7)
    st_ = LIB.fsdp_auto_wrap(n, backward, ag, rs, t, m, *a, mem_max, bucket_of if out else None,
                             ctypes.byref(nbv) if nb else None)
    return st_, list(bucket_of)[:max(n, 1)], nbv.value


def test_error_paths_leave_outputs_untouched():
    nan, inf = float("nan"), float("inf")
    cases = [
        (dict(n=-1), INVALID),
        (dict(n=3, backward=2), INVALID),
        (dict(n=3, ag=[1, -1, 1]), INVALID),
        (dict(n=3, backward=1, rs=[1, 1, -5]), INVALID),
        (dict(n=3, backward=1, rs="null"), INVALID),
        (dict(n=3, t=[1.0, nan, 1.0]), INVALID),
        (dict(n=3, t=[1.0, inf, 1.0]), INVALID),
        (dict(n=3, t=[1.0, -1.0, 1.0]), INVALID),
        (dict(n=3, m=[1, 1, -1]), INVALID),
        (dict(n=3, a=(-1.0, 0.0, 0.0, 0.0)), INVALID),
        (dict(n=3, a=(0.0, nan, 0.0, 0.0)), INVALID),
        (dict(n=3, a=(0.0, 0.0, 0.0, inf)), INVALID),
        (dict(n=3, mem_max=-1), INVALID),
        (dict(n=3, out=False), INVALID),
        (dict(n=3, ag=[1 << 52, 1 << 52, 1]), OVERFLOW),
        (dict(n=3, backward=1, rs=[1 << 53, 1, 0]), OVERFLOW),
        (dict(n=3, m=[(1 << 63) - 1, 1, 0]), OVERFLOW),
    ]
    for kw, want in cases:
        st_, out, nb = _raw(**kw)
        assert st_ == want, kw
        assert out == [-7] * len(out) and nb == -7, kw
        assert LIB.fsdp_last_error()
    st_, _, _ = _raw(3, nb=False)
    assert st_ == INVALID


def test_forward_ignores_rs_words_and_empty_pass():
    st_, out, nb = _raw(3, backward=0, rs="null")
    assert st_ == 0 and nb >= 1
    st_, out, nb = _raw(0)
    assert st_ == 0 and nb == 0
    assert auto_wrap([], [], [], 1.0, 1.0, 0) == []
    with pytest.raises(FsdpError):
        auto_wrap([1], [float("nan")], [0], 0.0, 0.0, 0)
    with pytest.raises(ValueError):
        auto_wrap([1, 2], [1.0], [0, 0], 0.0, 0.0, 0)
