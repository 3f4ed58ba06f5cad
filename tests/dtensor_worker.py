"""Worker for the DTensor pin: runs the paper's redistribute statement on gloo.

Each rank loads its inputs from ``workdir``, performs, per parameter,
``Shard(0) -> Replicate`` with ``forward_dtype=bfloat16`` and the backward
``Partial("avg") -> Shard(0)`` with ``backward_dtype=float32`` exactly as the
paper's ``replicate_compute`` listing states it (section 4), and saves the
results for the parent test to compare with the oracle.  With ``mixed=False``
both dtypes are fp32 (training without mixed precision) and the gradients
are fp32.
"""

import os

import numpy as np
import torch
import torch.distributed as dist
from torch.distributed.device_mesh import init_device_mesh
from torch.distributed.tensor import Partial, Replicate, Shard, distribute_tensor


def run(rank, world_size, port, workdir, num_params, mixed=True):
    os.environ["MASTER_ADDR"] = "127.0.0.1"
    os.environ["MASTER_PORT"] = str(port)
    dist.init_process_group("gloo", rank=rank, world_size=world_size)
    try:
        mesh = init_device_mesh("cpu", (world_size,))
        for p in range(num_params):
            x = torch.from_numpy(np.load(os.path.join(workdir, f"x_{p}.npy")))
            g = torch.from_numpy(np.load(os.path.join(workdir, f"g_{p}_{rank}.npy")))
            g = g.view(torch.bfloat16) if mixed else g.view(torch.float32)
            param = torch.nn.Parameter(distribute_tensor(x, mesh, [Shard(0)]))
            full = param.redistribute(
                placements=(Replicate(),),
                forward_dtype=torch.bfloat16 if mixed else torch.float32,
                backward_dtype=torch.float32,
            ).to_local(grad_placements=(Partial(reduce_op="avg"),))
            full.backward(g)
            view = torch.int16 if mixed else torch.int32
            np.save(os.path.join(workdir, f"ag_{p}_{rank}.npy"), full.detach().view(view).numpy())
            np.save(os.path.join(workdir, f"rs_{p}_{rank}.npy"), param.grad.to_local().numpy())
    finally:
        dist.destroy_process_group()
