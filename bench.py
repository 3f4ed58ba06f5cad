"""Benchmark: one rank's bucketed FSDP copy path on one MI355X.

A step is one pass of the whole hot path over one bucket (one transformer
block) at one rank (rank 0 unless --rank says otherwise):

    ag_pack (fp32 shards -> bf16 chunk, written into the rank's slot of the
    gathered buffer), ag_unpack (gathered W*S -> full bf16 params),
    rs_pack (full bf16 grads -> W*S send buffer), rs_reduce (W*S received
    chunks -> fp32 grad shards).

Inputs are seeded synthetic tensors of the workload's shapes and value
distributions (params N(0, 0.02) with RMSNorm weights 1.0, grads N(0, 1e-3)
in bf16), generated on the device before timing and resident in HBM.  The
metric is effective HBM bandwidth: the algorithmic bytes of the step (what
the method must read and write, padding writes included) divided by the
step time.  Per-kernel launch durations come from HIP events recorded on the
stream the kernels run on; the dominant kernel's figure is the roofline
entry.  A plain device-to-device copy of the unpack's bytes is timed beside
them as the achievable reference.  The CPU oracle is timed on a bounded
sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 3] [--rank 0]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective HBM GB/s (and % of peak) for bucket pack/unpack/reduce"
PEAK_GBPS = 8000.0                       # MI355X HBM3E
KERNELS = ("ag_pack", "ag_unpack", "rs_pack", "rs_reduce")
# device symbols of the kernels each call launches (bf16 wire, one contiguous
# buffer); rocprofv3 reports them by these names.  A small rank shard (fewer
# than 4 full-size tiles per CU) reduces with 128-thread workgroups instead.
KERNEL_SYMBOLS = {
    "ag_pack": "ag_pack_kernel<1, OneChunk>",
    "ag_unpack": "ag_unpack_kernel<ContigChunks>",
    "rs_pack": "rs_pack_kernel<ContigChunks, 0>",
    "rs_reduce": "rs_reduce_kernel<ContigChunks, unsigned short, 256>",
}
KERNEL_SOURCE = os.path.join(ROOT, "paper_2411_00284_amd", "csrc", "bucket_kernels.hip")
PROFILES = os.path.join(ROOT, "profiles")


def algorithmic_bytes(W, S, E, V0):
    """Bytes each kernel must move (padding zero-writes included)."""
    return {
        "ag_pack": 4 * V0 + 2 * S,
        "ag_unpack": 2 * E + 2 * E,
        "rs_pack": 2 * E + 2 * W * S,
        "rs_reduce": 2 * W * V0 + 4 * V0,
    }


def kernel_source_sha():
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def read_profile_avg_us(kernel: str, workload: str):
    """The kernel's average duration in the committed rocprofv3 summary of the
    same workload, or None when there is none or the kernel source changed
    since it was taken (event timing reads short kernels long; this is the
    kernel's own duration)."""
    path = os.path.join(PROFILES, f"kernels_{workload}_stats.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    if not m or m.group(1) != kernel_source_sha():
        return None
    m = re.search(rf"^\|\s*{kernel}\s*\|[^|]*\|[^|]*\|\s*([0-9.]+)\s*\|", text, re.M)
    return float(m.group(1)) if m else None


def read_traffic(kernel: str, workload: str):
    """HBM traffic per launch from the committed counter summary, or None when
    there is none or the kernel source changed since the counters were taken."""
    path = os.path.join(PROFILES, f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", text)
    if not m or m.group(1) != kernel_source_sha():
        return None
    m = re.search(rf"^\|\s*{kernel}\s*\|[^|]*\|[^|]*\|[^|]*\|\s*([0-9.eE+]+)\s*\|", text, re.M)
    return float(m.group(1)) if m else None


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, help="1 toy, 2 8B, 3 70B (default), 4 405B, 5 uneven, 6 70B TP-8 shards, 7 8B at W=128")
    ap.add_argument("--rank", type=int, default=0, help="the rank whose share is timed (0 <= rank < W)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip timing the fp32-wire and chunk-table forms after the steps")
    ap.add_argument("--variant-reps", type=int, default=10)
    ap.add_argument("--event-every", type=int, default=5,
                    help="record the per-kernel HIP events on every N-th timed step (N=1: every step)")
    ap.add_argument("--copy-cost", action="store_true",
                    help="also fit the alpha + beta*bytes copy cost over sub-buckets of the block "
                         "(launches the path kernels at other sizes, so it is off in profiled runs)")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step replayed from a HIP graph")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after the steps, run a plain 1 GiB device copy (for counter scaling)")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py: one GPU only (asked for --gpus {args.gpus}); "
              "the path has no collective and runs per rank", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2411_00284_amd import BucketPlan
    from synth import workload

    wl = workload(args.workload)
    W, rank = wl.world_size, args.rank
    if not 0 <= rank < W:
        print(f"bench.py: --rank {rank} is outside 0..{W - 1} for {wl.name}", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    plan = BucketPlan(W, wl.dims)
    S = plan.chunk_elems
    P = wl.num_params
    E = wl.total_elems
    V0 = sum(plan.local_elems(p, rank) for p in range(P))

    # ---- seeded synthetic inputs, resident in HBM before timing
    g = torch.Generator(device=dev)
    g.manual_seed(1000 + args.workload)

    def normal(n, scale, dtype):
        out = torch.empty(n, dtype=dtype, device=dev)
        step_n = 1 << 27
        for s in range(0, n, step_n):
            e = min(n, s + step_n)
            out[s:e] = (torch.randn(e - s, generator=g, device=dev) * scale).to(dtype)
        return out

    shards = []
    for p, (n, k) in enumerate(wl.dims):
        v = plan.local_elems(p, rank)
        shards.append(torch.ones(v, device=dev) if wl.is_norm[p] else normal(v, 0.02, torch.float32))
    gathered = normal(W * S, 0.02, torch.bfloat16)          # the other ranks' chunks
    send_chunk = gathered[rank * S:(rank + 1) * S]           # the rank packs into its own slot
    params = [torch.empty(n * k, dtype=torch.bfloat16, device=dev) for n, k in wl.dims]
    grads = [normal(n * k, 1e-3, torch.bfloat16) for n, k in wl.dims]
    send_buf = torch.empty(W * S, dtype=torch.bfloat16, device=dev)
    recv = normal(W * S, 1e-3, torch.bfloat16)
    outs = [torch.empty(plan.local_elems(p, rank), dtype=torch.float32, device=dev) for p in range(P)]
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()

    def run_step(ev=None, st=None):
        st = stream if st is None else st
        if ev is not None:
            ev[0].record(st)
        plan.ag_pack(rank, shards, send_chunk, st)
        if ev is not None:
            ev[1].record(st)
        plan.ag_unpack(gathered, params, st)
        if ev is not None:
            ev[2].record(st)
        plan.rs_pack(grads, send_buf, st)
        if ev is not None:
            ev[3].record(st)
        plan.rs_reduce(rank, recv, outs, st)
        if ev is not None:
            ev[4].record(st)

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()

    # Every step is timed by the wall clock; the per-kernel events (each record
    # adds a marker packet between the kernels) go on every N-th step only.
    every = max(1, args.event_every)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] if k % every == 0 else None
              for k in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        run_step(events[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    per_kernel_ms = {name: [] for name in KERNELS}
    for ev in events:
        if ev is None:
            continue
        for i, name in enumerate(KERNELS):
            per_kernel_ms[name].append(ev[i].elapsed_time(ev[i + 1]))
    abytes = algorithmic_bytes(W, S, E, V0)
    step_bytes = sum(abytes.values())
    kernels = {}
    for name in KERNELS:
        avg_ms = float(np.mean(per_kernel_ms[name]))
        gbps = abytes[name] / (avg_ms * 1e-3) / 1e9
        kernels[name] = {"avg_us": round(avg_ms * 1e3, 2),
                         "median_us": round(float(np.median(per_kernel_ms[name])) * 1e3, 2),
                         "min_us": round(float(np.min(per_kernel_ms[name])) * 1e3, 2),
                         "bytes": abytes[name], "GBps": round(gbps, 1), "frac": round(gbps / PEAK_GBPS, 4),
                         "rocprof_avg_us": read_profile_avg_us(name, wl.name)}

    copy_ref = None if args.no_variants else time_d2d_copy(gathered, send_buf, stream, args.variant_reps)

    variants = None if args.no_variants else time_variants(
        plan, wl, rank, shards, gathered, params, grads, send_buf, recv, outs, stream, args.variant_reps)

    if args.copy_probe:
        n = 1 << 29                                # 1 GiB of bf16 read, 1 GiB written
        a = torch.empty(n, dtype=torch.bfloat16, device=dev)
        b = torch.empty_like(a)
        a.fill_(1.0)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    dominant = max(KERNELS, key=lambda n: kernels[n]["avg_us"])
    dom = kernels[dominant]
    roofline = {
        "bound": "hbm",
        "kernel": KERNEL_SYMBOLS[dominant],
        "achieved": dom["GBps"],
        "peak": PEAK_GBPS,
        "unit": "GB/s",
        "frac": dom["frac"],
        "traffic": read_traffic(dominant, wl.name),
    }

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, rank, gpu_plan=plan)

    ms_per_step = elapsed / args.steps * 1e3
    line = {
        "metric": METRIC,
        "value": round(step_bytes / (elapsed / args.steps) / 1e9, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "world_size": W, "rank": rank, "params": P, "chunk_elems": S,
                   "block_elems": E, "rank_elems": V0, "align_elems": 8, "wire": "bf16",
                   "step": "ag_pack+ag_unpack+rs_pack+rs_reduce", "step_bytes": step_bytes},
        "frac_of_peak": round(step_bytes / (elapsed / args.steps) / 1e9 / PEAK_GBPS, 4),
        "kernels": kernels,
        "kernel_event_steps": len(per_kernel_ms[KERNELS[0]]),
        "roofline": roofline,
        "d2d_copy": copy_ref,
        "cpu_baseline": cpu,
        "variants": variants,
        "auto_wrap": None if args.no_variants else time_auto_wrap(wl),
        "copy_cost": fit_copy_cost(wl, stream) if args.copy_cost else None,
        "graph": None if not args.graph else time_graph_step(
            lambda: run_step(None, torch.cuda.current_stream()), args.steps),
    }
    print(json.dumps(line), flush=True)
    plan.close()
    return 0


def time_d2d_copy(src, dst, stream, reps):
    """A plain device-to-device copy of ``src`` into ``dst`` (torch ``copy_``
    of two contiguous same-type tensors, which is the runtime's
    hipMemcpyAsync), timed with HIP events on ``stream``: the achievable
    reference for the copy kernels, at the unpack's bytes."""
    import numpy as np
    import torch

    nbytes = 2 * src.numel() * src.element_size()
    with torch.cuda.stream(stream):
        dst.copy_(src)
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        with torch.cuda.stream(stream):
            dst.copy_(src)
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b))
    avg_ms = float(np.mean(times))
    gbps = nbytes / (avg_ms * 1e-3) / 1e9
    return {"kind": "hipMemcpyAsync device to device (torch copy_)", "bytes": nbytes,
            "avg_us": round(avg_ms * 1e3, 2), "median_us": round(float(np.median(times)) * 1e3, 2),
            "GBps": round(gbps, 1), "frac": round(gbps / PEAK_GBPS, 4)}


def time_variants(plan, wl, rank, shards, gathered, params, grads, send_buf, recv, outs, stream, reps):
    """Average launch time of the element-type and chunk-table forms, on the
    same bucket: fp32 and fp16 param_dtype packs, the pack pushed to W chunks,
    W-chunk-table unpack / pack / reduce
    (tables pointing into the same buffers), bf16 gradients cast to an fp32
    wire, and the fp32 and fp16 reduces."""
    import numpy as np
    import torch

    W, S = wl.world_size, plan.chunk_elems
    E = wl.total_elems
    V0 = sum(plan.local_elems(p, rank) for p in range(wl.num_params))
    dev = recv.device
    send_chunk32 = torch.empty(S, dtype=torch.float32, device=dev)
    send32 = torch.empty(W * S, dtype=torch.float32, device=dev)
    recv32 = torch.empty(W * S, dtype=torch.float32, device=dev)
    recv32.copy_(recv)                                  # the same values, widened
    g_chunks = [gathered[i * S:(i + 1) * S] for i in range(W)]
    s_chunks = [send_buf[i * S:(i + 1) * S] for i in range(W)]
    r_chunks = [recv[i * S:(i + 1) * S] for i in range(W)]
    s32_chunks = [send32[i * S:(i + 1) * S] for i in range(W)]
    r32_chunks = [recv32[i * S:(i + 1) * S] for i in range(W)]
    send_chunk16 = torch.empty(S, dtype=torch.float16, device=dev)
    recv16 = recv.view(torch.float16)                   # the same bytes read as fp16 (timing only)
    r16_chunks = [recv16[i * S:(i + 1) * S] for i in range(W)]
    cases = {
        "ag_pack_f32": (lambda: plan.ag_pack_ex(rank, shards, send_chunk32, "f32", stream), 4 * V0 + 4 * S),
        "ag_pack_f16": (lambda: plan.ag_pack_ex(rank, shards, send_chunk16, "f16", stream), 4 * V0 + 2 * S),
        "ag_pack_push": (lambda: plan.ag_pack_push(rank, shards, s_chunks, "bf16", stream), 4 * V0 + 2 * W * S),
        "ag_unpack_chunks": (lambda: plan.ag_unpack_ex(g_chunks, params, "bf16", stream), 4 * E),
        "rs_pack_chunks": (lambda: plan.rs_pack_ex(grads, s_chunks, "bf16", stream), 2 * E + 2 * W * S),
        "rs_pack_bf16_to_f32": (lambda: plan.rs_pack_ex(grads, s32_chunks, "f32", stream), 2 * E + 4 * W * S),
        "rs_reduce_chunks": (lambda: plan.rs_reduce_ex(rank, r_chunks, outs, "bf16", stream), 2 * W * V0 + 4 * V0),
        "rs_reduce_f32": (lambda: plan.rs_reduce_ex(rank, r32_chunks, outs, "f32", stream), 4 * W * V0 + 4 * V0),
        "rs_reduce_f16": (lambda: plan.rs_reduce_ex(rank, r16_chunks, outs, "f16", stream), 2 * W * V0 + 4 * V0),
    }
    flush = torch.empty(1 << 28, dtype=torch.int32, device=dev)   # 1 GiB: evicts L2 and the 256 MB MALL
    res = {}
    for name, (fn, nbytes) in cases.items():
        fn()
        torch.cuda.synchronize()
        times = []
        for k in range(reps):
            flush.fill_(k)
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            b.synchronize()
            times.append(a.elapsed_time(b))
        avg_ms = float(np.mean(times))
        gbps = nbytes / (avg_ms * 1e-3) / 1e9
        res[name] = {"avg_us": round(avg_ms * 1e3, 2), "bytes": nbytes, "GBps": round(gbps, 1),
                     "frac": round(gbps / PEAK_GBPS, 4)}
    del send_chunk32, send32, recv32, send_chunk16, flush
    return res


def time_auto_wrap(wl, layers=80, reps=20):
    """Host time of the library's auto-wrapping planner (fsdp_auto_wrap) on a
    whole-model pass: ``layers`` copies of the workload's block, one node per
    parameter.  Node words are the padded all-gather sizes at the workload's W;
    compute times and memories are a synthetic scale (2 flop per weight and
    token over 65536 tokens at 2.5 PFLOP/s; bf16 weights plus a fixed
    activation share), and the collectives cost 20 us + 2 bytes / 100 GB/s per
    word.  Only the planner is timed (binding included)."""
    import numpy as np

    from paper_2411_00284_amd import auto_wrap

    W = wl.world_size
    ag, t, m = [], [], []
    for _ in range(layers):
        for n, k in wl.dims:
            ag.append(W * (-(-n // W)) * k)
            t.append(2.0 * n * k * 65536 / 2.5e15)
            m.append(2 * n * k + (1 << 24))
    res = {"nodes": len(ag)}
    for name, backward in (("forward", False), ("backward", True)):
        times = []
        for _ in range(reps):
            t0 = time.perf_counter()
            buckets = auto_wrap(ag, t, m, 20e-6, 2 / 100e9, 8 << 30, backward, ag, 20e-6, 2 / 100e9)
            times.append(time.perf_counter() - t0)
        res[name] = {"buckets": len(buckets), "us_per_pass": round(float(np.median(times)) * 1e6, 1)}
    return res


def time_graph_step(run_step, steps):
    """The same step captured once in a HIP graph (torch.cuda.CUDAGraph) and
    replayed ``steps`` times back to back: wall time per step.  The four calls
    allocate nothing and make no memset, so they can be captured; the replay
    removes the host launch cost, which matters only for small buckets."""
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run_step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run_step()
    graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        graph.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / steps * 1e3
    del graph
    return {"ms_per_step": round(ms, 4)}


def fit_copy_cost(wl, stream, reps=5):
    """Copy-in + copy-out cost of a bucket as a function of its size, on this
    GPU: buckets made of subsets of the workload's block (one norm up to the
    whole block) are timed for the forward pair (ag_pack + ag_unpack) and the
    backward pair (rs_pack + rs_reduce), with a 1 GiB cache flush before each
    rep, and T = alpha + beta * bytes is fitted by least squares over the
    algorithmic bytes of the pair.  This is the measured copy part of the
    alpha-beta model that auto-wrapping prices buckets with."""
    import numpy as np
    import torch

    from paper_2411_00284_amd import BucketPlan

    W = wl.world_size
    names = list(wl.names)
    sets = [[len(names) - 1], [1], [1, 2], [0], [0, 1, 2, 3], [4], [4, 5, 6], list(range(len(names)))]
    dev = torch.device("cuda:0")
    flush = torch.empty(1 << 28, dtype=torch.int32, device=dev)
    pts = {"forward": [], "backward": []}
    for sel in sets:
        dims = [wl.dims[p] for p in sel]
        plan = BucketPlan(W, dims)
        S = plan.chunk_elems
        V0 = sum(plan.local_elems(p, 0) for p in range(len(dims)))
        E = sum(n * k for n, k in dims)
        shards = [torch.zeros(plan.local_elems(p, 0), device=dev) for p in range(len(dims))]
        gathered = torch.zeros(W * S, dtype=torch.bfloat16, device=dev)
        params = [torch.empty(n * k, dtype=torch.bfloat16, device=dev) for n, k in dims]
        outs = [torch.empty(plan.local_elems(p, 0), device=dev) for p in range(len(dims))]
        pairs = {
            "forward": (lambda: (plan.ag_pack(0, shards, gathered[:S], stream),
                                 plan.ag_unpack(gathered, params, stream)), 4 * V0 + 2 * S + 4 * E),
            "backward": (lambda: (plan.rs_pack(params, gathered, stream),
                                  plan.rs_reduce(0, gathered, outs, stream)), 2 * E + 2 * W * S + 2 * W * V0 + 4 * V0),
        }
        for name, (fn, nbytes) in pairs.items():
            fn()
            torch.cuda.synchronize()
            times = []
            for k in range(reps):
                flush.fill_(k)
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record(stream)
                fn()
                b.record(stream)
                b.synchronize()
                times.append(a.elapsed_time(b) * 1e3)
            pts[name].append((nbytes, float(np.median(times))))
        plan.close()
        del shards, gathered, params, outs
    del flush
    res = {}
    for name, xy in pts.items():
        x = np.array([p[0] for p in xy], dtype=np.float64)
        y = np.array([p[1] for p in xy], dtype=np.float64)
        beta, alpha = np.polyfit(x, y, 1)
        pred = alpha + beta * x
        r2 = 1.0 - float(np.sum((y - pred) ** 2) / np.sum((y - y.mean()) ** 2))
        res[name] = {"alpha_us": round(float(alpha), 2), "GBps": round(1e-3 / float(beta), 1),
                     "r2": round(r2, 5), "points": [[int(a), round(b, 2)] for a, b in xy]}
    return res


def cpu_baseline(wl, rank=0, min_seconds=10.0, max_passes=50, gpu_plan=None):
    """The oracle, as it stands, timed on the host: all four steps at ``rank``
    over the whole bucket, repeated until about ``min_seconds`` of CPU work
    has been measured (the oracle is single-threaded numpy).  With
    ``gpu_plan`` (the library's plan of the same bucket) the four library
    calls then run once on the same inputs and their outputs are compared with
    the oracle's, bit for bit: the record's parity verdict."""
    import numpy as np

    import oracle.fsdp_oracle as O
    from synth import random_bits16, random_bits32

    dims = list(wl.dims)
    W = wl.world_size
    plan = O.make_plan(W, dims, 8)
    S = plan.chunk
    E = sum(n * k for n, k in dims)
    V0 = sum(O.local_elems(plan, p, rank) for p in range(len(dims)))
    shards = [random_bits32([1, p], O.local_elems(plan, p, rank)).view(np.float32) for p in range(len(dims))]
    shards = [np.where(np.isfinite(s), s, np.float32(0)) for s in shards]
    gathered = random_bits16([2], W * S)
    grads = [random_bits16([3, p], n * k).reshape(n, k) for p, (n, k) in enumerate(dims)]
    recv = (random_bits16([4], W * S) & np.uint16(0xBFFF))      # finite: exponent MSB cleared
    t = {k: 0.0 for k in ("ag_pack", "ag_unpack", "rs_pack", "rs_reduce")}
    passes = 0
    while passes < max_passes and (passes == 0 or sum(t.values()) < min_seconds):
        t0 = time.perf_counter(); want_pack = O.ag_pack(plan, rank, shards); t["ag_pack"] += time.perf_counter() - t0
        t0 = time.perf_counter(); want_unpack = O.ag_unpack(plan, gathered); t["ag_unpack"] += time.perf_counter() - t0
        t0 = time.perf_counter(); want_send = O.rs_pack(plan, grads); t["rs_pack"] += time.perf_counter() - t0
        t0 = time.perf_counter(); want_red = O.rs_reduce(plan, rank, recv); t["rs_reduce"] += time.perf_counter() - t0
        passes += 1
    parity = None
    if gpu_plan is not None:
        parity = library_parity(gpu_plan, rank, shards, gathered, grads, recv,
                                (want_pack, want_unpack, want_send, want_red))
        del want_pack, want_unpack, want_send, want_red
    b = algorithmic_bytes(W, S, E, V0)
    total_s = sum(t.values())
    return {
        "value": round(passes * sum(b.values()) / total_s / 1e9, 3),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{wl.name}: the whole bucket ({len(dims)} params, W={W}, {sum(b.values())} algorithmic "
                   f"bytes per pass), all four steps at rank {rank}, {passes} passes, numpy single thread; "
                   f"host has {len(os.sched_getaffinity(0))} cores"),
        "seconds": round(total_s, 3),
        "per_pass_s": {k: round(v / passes, 4) for k, v in t.items()},
        "parity": parity,
    }


def library_parity(plan, rank, shards, gathered, grads, recv, want):
    """Each library call once on the oracle's inputs: does every output element
    equal the oracle's, bit for bit?"""
    import numpy as np
    import torch

    dev = torch.device("cuda:0")

    def up16(a):
        return torch.from_numpy(np.ascontiguousarray(a).reshape(-1).view(np.int16)).to(dev).view(torch.bfloat16)

    def down(t, dtype):
        return t.view(torch.int16 if dtype == np.uint16 else torch.int32).cpu().numpy().view(dtype)

    want_pack, want_unpack, want_send, want_red = want
    P, S, W = plan.num_params, plan.chunk_elems, plan.world_size
    res = {}
    d_shards = [torch.from_numpy(np.ascontiguousarray(x)).to(dev) for x in shards]
    out = torch.empty(S, dtype=torch.bfloat16, device=dev)
    plan.ag_pack(rank, d_shards, out)
    res["ag_pack"] = bool(np.array_equal(down(out, np.uint16), want_pack))
    del d_shards, out
    d_gathered = up16(gathered)
    params = [torch.empty(plan.full_elems(p), dtype=torch.bfloat16, device=dev) for p in range(P)]
    plan.ag_unpack(d_gathered, params)
    res["ag_unpack"] = all(np.array_equal(down(params[p], np.uint16), want_unpack[p].reshape(-1)) for p in range(P))
    del d_gathered, params
    d_grads = [up16(g) for g in grads]
    send = torch.empty(W * S, dtype=torch.bfloat16, device=dev)
    plan.rs_pack(d_grads, send)
    res["rs_pack"] = bool(np.array_equal(down(send, np.uint16), want_send))
    del d_grads, send
    d_recv = up16(recv)
    outs = [torch.empty(plan.local_elems(p, rank), dtype=torch.float32, device=dev) for p in range(P)]
    plan.rs_reduce(rank, d_recv, outs)
    res["rs_reduce"] = all(np.array_equal(down(outs[p], np.uint32), want_red[p].reshape(-1).view(np.uint32))
                           for p in range(P))
    del d_recv, outs
    torch.cuda.empty_cache()
    return res


if __name__ == "__main__":
    sys.exit(main())
