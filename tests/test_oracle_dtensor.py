"""The oracle against torch's DTensor running the paper's redistribute statement.

The paper defines the forward all-gather and the backward reduce-scatter of
SimpleFSDP through ``DTensor.redistribute`` (section 3.1; section 4,
``replicate_compute``).  Here that exact statement runs on W gloo processes
on the CPU, one parameter at a time (no bucket), and the oracle's bucketed
path (pack, exchange, unpack; pack, exchange, reduce) must reproduce it:

* all-gather: bit-exact for arbitrary fp32 values (torch's bf16 cast and the
  oracle's are both round-half-to-even);
* reduce-scatter average: bit-exact whenever the fp32 sum is order-free,
  i.e. for W = 2 with arbitrary values and for any W with values whose sums
  are exact (torch's average is then one correctly rounded division by W).

Both the mixed-precision setting (bf16 all-gather, bf16 gradients reduced in
fp32) and the plain fp32 setting are run; for the former the oracle's fp32
reduce-scatter wire must also agree.
"""

import os
import socket

import numpy as np
import pytest
import torch.multiprocessing as mp

import oracle.fsdp_oracle as O
from synth import exact_grad_bits, random_bits32

import dtensor_worker

DIMS = [(7, 3), (1, 5), (2, 1), (13, 4), (4, 2)]


def _free_port():
    with socket.socket() as s:
        s.bind(("127.0.0.1", 0))
        return s.getsockname()[1]


def _oracle_all_gather(plan, xs, param_dtype="bf16"):
    chunks = []
    for r in range(plan.world_size):
        local = []
        for p, x in enumerate(xs):
            c = plan.rows_per_rank[p]
            n = O.local_rows(plan, p, r)
            local.append(x[r * c:r * c + n])
        chunks.append(O.ag_pack(plan, r, local, param_dtype))
    return O.ag_unpack(plan, O.all_gather(chunks))


def _oracle_reduce_scatter(plan, grads_by_rank, reduce_dtype=None):
    sends = [O.rs_pack(plan, g, reduce_dtype) for g in grads_by_rank]
    return [O.rs_reduce(plan, j, O.rs_exchange(sends, j, plan.chunk)) for j in range(plan.world_size)]


@pytest.mark.slow
@pytest.mark.parametrize("w,exact,mixed", [(2, False, True), (3, True, True), (5, True, True),
                                           (2, False, False), (3, True, False)])
def test_oracle_matches_dtensor(tmp_path, w, exact, mixed):
    rng_words = [w, int(exact), int(mixed)]
    xs = []
    for p, (n, k) in enumerate(DIMS):
        x = random_bits32(rng_words + [p], n * k).view(np.float32).reshape(n, k).copy()
        x[np.isnan(x)] = 1.5          # torch and the oracle may pick different NaN payloads
        xs.append(x)
        np.save(tmp_path / f"x_{p}.npy", x)
    grads = []
    for r in range(w):
        gr = []
        for p, (n, k) in enumerate(DIMS):
            if exact:
                g = exact_grad_bits(rng_words + [r, p], (n, k))
            else:
                f = np.random.default_rng(rng_words + [r, p]).standard_normal((n, k)) \
                    * np.exp2(np.random.default_rng(rng_words + [r, p, 1]).integers(-20, 21, (n, k)))
                g = (f.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
            if not mixed:
                g = O.bf16_to_f32(g).reshape(n, k)         # fp32 gradients with the same values
                if not exact:
                    g = g * np.float32(1.0 + 2.0 ** -20)     # use bits below bf16 precision too
            gr.append(g)
            np.save(tmp_path / f"g_{p}_{r}.npy", g.view(np.int16) if mixed else g.view(np.int32))
        grads.append(gr)

    mp.spawn(dtensor_worker.run, args=(w, _free_port(), str(tmp_path), len(DIMS), mixed), nprocs=w, join=True)

    plan = O.make_plan(w, DIMS, 8)
    ag = _oracle_all_gather(plan, xs, "bf16" if mixed else "f32")
    rs_variants = [_oracle_reduce_scatter(plan, grads)]
    if mixed:
        rs_variants.append(_oracle_reduce_scatter(plan, grads, "f32"))
    for p in range(len(DIMS)):
        for r in range(w):
            got = np.load(tmp_path / f"ag_{p}_{r}.npy")
            want = ag[p].view(np.uint16) if mixed else ag[p].view(np.uint32)
            assert np.array_equal(got.view(want.dtype), want), (p, r)
            got_rs = np.load(tmp_path / f"rs_{p}_{r}.npy")
            for rs in rs_variants:
                assert got_rs.shape == rs[r][p].shape, (p, r)
                assert np.array_equal(got_rs.view(np.uint32), rs[r][p].view(np.uint32)), (p, r)
