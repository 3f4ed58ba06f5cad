"""The four hot calls captured in a HIP graph (through torch.cuda.CUDAGraph)
and replayed: every replay reproduces the eagerly launched step bit for bit,
and the toy block's replay also equals the oracle.

The calls allocate nothing, make no memset and enqueue one kernel each on the
current stream, so they can be captured.  Between replays the outputs are
poisoned by eager fill kernels and the host synchronises, as a training loop
would run other work between steps.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle.fsdp_oracle as O
from gpu_util import DEV, dev_random_bits16, dev_wide_bf16, host_u16, host_u32, step
from synth import WORKLOADS

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

if torch.cuda.is_available():
    from paper_2411_00284_amd import BucketPlan


def _bits(t):
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


@pytest.mark.parametrize("key", [1, 2, 5])
def test_step_replayed_from_a_graph(key):
    wl = WORKLOADS[key]
    W = wl.world_size
    rank = W - 1
    plan = BucketPlan(W, wl.dims)
    S = plan.chunk_elems
    P = wl.num_params
    g = torch.Generator(device=DEV)
    g.manual_seed(key)
    shards = [torch.randn(plan.local_elems(p, rank), device=DEV, generator=g) for p in range(P)]
    gathered = dev_random_bits16(W * S, 10 + key)
    params = [torch.empty(n * k, dtype=torch.bfloat16, device=DEV) for n, k in wl.dims]
    grads = [dev_random_bits16(n * k, 20 + key + p) for p, (n, k) in enumerate(wl.dims)]
    send_buf = torch.empty(W * S, dtype=torch.bfloat16, device=DEV)
    recv = dev_wide_bf16(W * S, 30 + key)
    outs = [torch.empty(plan.local_elems(p, rank), dtype=torch.float32, device=DEV) for p in range(P)]
    outputs = [gathered[rank * S:(rank + 1) * S], *params, send_buf, *outs]

    def one_step():
        plan.ag_pack(rank, shards, gathered[rank * S:(rank + 1) * S])
        plan.ag_unpack(gathered, params)
        plan.rs_pack(grads, send_buf)
        plan.rs_reduce(rank, recv, outs)

    step(f"graph: eager step {wl.name}")
    one_step()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outputs]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        one_step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    step(f"graph: capture {wl.name}")
    with torch.cuda.graph(graph):
        one_step()
    torch.cuda.synchronize()
    for rep in range(3):
        for o in outputs:
            o.view(torch.uint8).fill_(0xFF)
        torch.cuda.synchronize()
        step(f"graph: replay {rep} {wl.name}")
        graph.replay()
        torch.cuda.synchronize()
        for i, (o, r) in enumerate(zip(outputs, ref)):
            assert torch.equal(_bits(o), _bits(r)), (rep, i)

    if key == 1:
        oplan = O.make_plan(W, wl.dims)
        host_shards = [host_u32(s).view(np.float32) for s in shards]
        assert np.array_equal(host_u16(outputs[0]), O.ag_pack(oplan, rank, host_shards))
        want = O.ag_unpack(oplan, host_u16(gathered))
        for p in range(P):
            assert np.array_equal(host_u16(params[p]), want[p].reshape(-1))
        want = O.rs_pack(oplan, [host_u16(gr).reshape(n, k) for gr, (n, k) in zip(grads, wl.dims)])
        assert np.array_equal(host_u16(send_buf), want)
        want = O.rs_reduce(oplan, rank, host_u16(recv))
        for p in range(P):
            assert np.array_equal(host_u32(outs[p]), want[p].reshape(-1).view(np.uint32))
    del graph
    plan.close()


@pytest.mark.parametrize("W", [4, 8, 48])
def test_push_replayed_from_a_graph(W):
    """The push (one kernel below W = 8, a pack and a copy from W = 8 on; the
    copy takes its destinations in grid rows of 16 at W = 48) captured and
    replayed: every replay equals the eager push."""
    dims = [(3 * W + 1, 64), (W + 3, 1), (5, 8)]
    rank = W // 2
    plan = BucketPlan(W, dims)
    S = plan.chunk_elems
    g = torch.Generator(device=DEV)
    g.manual_seed(W)
    shards = [torch.randn(plan.local_elems(p, rank), device=DEV, generator=g) for p in range(len(dims))]
    dsts = [torch.empty(S, dtype=torch.bfloat16, device=DEV) for _ in range(W)]
    step(f"graph: eager push W={W}")
    plan.ag_pack_push(rank, shards, dsts)
    torch.cuda.synchronize()
    ref = [d.clone() for d in dsts]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        plan.ag_pack_push(rank, shards, dsts)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    step(f"graph: capture push W={W}")
    with torch.cuda.graph(graph):
        plan.ag_pack_push(rank, shards, dsts)
    torch.cuda.synchronize()
    for rep in range(3):
        for d in dsts:
            d.view(torch.uint8).fill_(0xFF)
        torch.cuda.synchronize()
        step(f"graph: replay {rep} push W={W}")
        graph.replay()
        torch.cuda.synchronize()
        for j, (d, r) in enumerate(zip(dsts, ref)):
            assert torch.equal(_bits(d), _bits(r)), (rep, j)
    del graph
    plan.close()
