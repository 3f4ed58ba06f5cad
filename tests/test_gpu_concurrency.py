"""One plan shared by several host threads, each launching the four calls on
its own stream (default priority) into its own buffers, many times over:
every thread's outputs stay bit-exact against the oracle."""

from __future__ import annotations

import threading

import numpy as np
import pytest
import torch

import oracle.fsdp_oracle as O
from gpu_util import DEV, host_u16, host_u32, step, to_dev_f32, to_dev_u16
from synth import WORKLOADS, random_bits16, random_bits32

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU"),
              pytest.mark.filterwarnings("ignore::RuntimeWarning")]

if torch.cuda.is_available():
    from paper_2411_00284_amd import BucketPlan


def test_threads_and_streams_share_a_plan():
    wl = WORKLOADS[1]
    W = wl.world_size
    dims = list(wl.dims)
    plan = BucketPlan(W, dims)
    oplan = O.make_plan(W, dims)
    S = oplan.chunk
    P = len(dims)
    nthreads, iters = 4, 25
    errors = []

    def worker(i):
        try:
            torch.cuda.set_device(DEV)
            stream = torch.cuda.Stream()            # default priority
            r = i % W
            shards_h = [random_bits32([70, i, p], O.local_elems(oplan, p, r)).view(np.float32) for p in range(P)]
            shards_h = [np.where(np.isfinite(s), s, np.float32(0)) for s in shards_h]
            gathered_h = random_bits16([71, i], W * S)
            grads_h = [random_bits16([72, i, p], n * k) for p, (n, k) in enumerate(dims)]
            recv_h = (random_bits16([73, i], W * S) & np.uint16(0xBFFF))      # finite values
            with torch.cuda.stream(stream):
                shards = [to_dev_f32(s) for s in shards_h]
                gathered = to_dev_u16(gathered_h)
                grads = [to_dev_u16(g) for g in grads_h]
                recv = to_dev_u16(recv_h)
                send = torch.empty(S, dtype=torch.bfloat16, device=DEV)
                params = [torch.empty(n * k, dtype=torch.bfloat16, device=DEV) for n, k in dims]
                send_buf = torch.empty(W * S, dtype=torch.bfloat16, device=DEV)
                outs = [torch.empty(O.local_elems(oplan, p, r), dtype=torch.float32, device=DEV) for p in range(P)]
                for _ in range(iters):
                    plan.ag_pack(r, shards, send, stream)
                    plan.ag_unpack(gathered, params, stream)
                    plan.rs_pack(grads, send_buf, stream)
                    plan.rs_reduce(r, recv, outs, stream)
            stream.synchronize()
            assert np.array_equal(host_u16(send), O.ag_pack(oplan, r, shards_h))
            want = O.ag_unpack(oplan, gathered_h)
            for p in range(P):
                assert np.array_equal(host_u16(params[p]), want[p].reshape(-1))
            want = O.rs_pack(oplan, [g.reshape(n, k) for g, (n, k) in zip(grads_h, dims)])
            assert np.array_equal(host_u16(send_buf), want)
            want = O.rs_reduce(oplan, r, recv_h)
            for p in range(P):
                assert np.array_equal(host_u32(outs[p]), want[p].reshape(-1).view(np.uint32))
        except Exception as e:   # noqa: BLE001 - reported below
            errors.append((i, e))

    step(f"concurrency: {nthreads} threads x {iters} steps, toy block")
    threads = [threading.Thread(target=worker, args=(i,)) for i in range(nthreads)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    plan.close()
    assert not errors, errors
