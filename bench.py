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
step time.  HIP events recorded on the stream the kernels run on time every
kernel inside the steps; the kernel with the longest launches gives the
roofline entry.  A per-kernel leg then launches each call 30 times over
rotating input/output sets of more than 1.5 GiB (so no launch finds its data
in the caches), with the device kept busy while the host enqueues them, and
reports the median and minimum by HIP events and, from a child run of the same
leg under a rocprofv3 kernel trace, by the kernels' own start and end
timestamps.  A plain device-to-device copy of the unpack's bytes is timed
beside them as the achievable reference.  The CPU oracle is timed on a
bounded sample of the same workload.

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
# Device symbols of the kernels each call launches (bf16 wire, one contiguous
# buffer), as rocprofv3 prints them; a kernel trace taken during the run
# replaces these with the names it saw.  A rank shard of fewer than 4
# full-size reduce tiles per CU is reduced with 128-thread workgroups; a
# single-chunk pack of fewer than 4 big (256-thread, 4-step) tiles per CU
# packs with 128-thread, 1-step tiles.
# The copies and the reduce have a second form ("true") that the library
# launches when some segment of the bucket is off the 16-byte grid.
KERNEL_SYMBOLS = {
    "ag_pack": "ag_pack_kernel<1, OneChunk, 256, 4>",
    "ag_unpack": "ag_unpack_kernel<ContigChunks, false>",
    "rs_pack": "rs_pack_kernel<ContigChunks, 0, false>",
    "rs_reduce": "rs_reduce_kernel<ContigChunks, unsigned short, 256, false>",
}
REDUCE_SMALL_SYMBOL = "rs_reduce_kernel<ContigChunks, unsigned short, 128, false>"
PACK_SMALL_SYMBOL = "ag_pack_kernel<1, OneChunk, 128, 1>"
KERNEL_BASENAMES = ("ag_pack_kernel", "ag_unpack_kernel", "rs_pack_kernel", "rs_reduce_kernel", "probe_read_kernel",
                    "probe_fill_kernel", "probe_copy_kernel", "probe_cast_kernel", "probe_reduce_kernel",
                    "probe_empty_kernel")
PROBES_LIB = os.path.join(ROOT, "paper_2411_00284_amd", "libfsdp_probes.so")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2411_00284_amd", "csrc", "bucket_kernels.hip")
PROFILES = os.path.join(ROOT, "profiles")
# The per-kernel leg cycles through input/output sets that together hold more
# than this many bytes, so that no launch finds its data in the L2 caches or
# the 256 MB Infinity Cache.
ROTATE_BYTES = 3 << 29
SLEEP_CYCLES = 50_000_000                # a device-side wait that lets the host enqueue a whole leg
# The full-size reduce tile, the big pack tile and the thresholds of the
# library's choice between the two shapes of each.
REDUCE_TILE = 256 * 8 * 2
SMALL_SHARD_TILES_PER_CU = 4
PACK_BIG_TILE = 256 * 8 * 4
PACK_SMALL_TILE = 128 * 8
PACK_BIG_TILES_PER_CU = 4


def algorithmic_bytes(W, S, E, V0):
    """Bytes each kernel must move (padding zero-writes included)."""
    return {
        "ag_pack": 4 * V0 + 2 * S,
        "ag_unpack": 2 * E + 2 * E,
        "rs_pack": 2 * E + 2 * W * S,
        "rs_reduce": 2 * W * V0 + 4 * V0,
    }


def kernel_symbol(name, plan, rank, cus):
    """The symbol the call launches for this plan and rank (bf16 wire, one
    contiguous bucket buffer, 16-byte-aligned tensors)."""
    P, S = plan.num_params, plan.chunk_elems
    off_grid = (2 * S) % 16 != 0 or any((2 * plan.offset(p)) % 16 for p in range(P))
    if name in ("ag_unpack", "rs_pack") and (off_grid or any((2 * plan.seg_elems(p)) % 16 for p in range(P))):
        return KERNEL_SYMBOLS[name].replace("false>", "true>")
    if name == "rs_reduce":
        full_tiles = sum(-(-plan.local_elems(p, rank) // REDUCE_TILE) for p in range(P))
        sym = REDUCE_SMALL_SYMBOL if full_tiles < SMALL_SHARD_TILES_PER_CU * cus else KERNEL_SYMBOLS[name]
        return sym.replace("false>", "true>") if off_grid else sym
    if name == "ag_pack":
        if pack_tiles(plan, PACK_BIG_TILE) < PACK_BIG_TILES_PER_CU * cus:
            return PACK_SMALL_SYMBOL
    return KERNEL_SYMBOLS[name]


def kernel_source_sha():
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def read_profile_avg_us(kernel: str, workload: str):
    """The kernel's average duration in the committed rocprofv3 summary of the
    same workload, or None when there is none or the kernel source changed
    since it was taken."""
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


def stats_us(ms_list):
    """Median, minimum and mean of launch times given in ms, in us."""
    import numpy as np
    a = np.asarray(ms_list, dtype=np.float64) * 1e3
    return {"median_us": round(float(np.median(a)), 3), "min_us": round(float(a.min()), 3),
            "mean_us": round(float(a.mean()), 3)}


# ----------------------------------------------------------------- per-kernel leg

def kernel_set(name, plan, wl, rank, dev, gen):
    """One input/output set of a kernel's call at ``rank``: returns the call
    (taking a stream) and the tensors it keeps alive.  Values follow the
    workload recipe (params N(0, 0.02), norms 1.0, bf16 N(0, 1e-3) grads)."""
    import torch

    S, W, P = plan.chunk_elems, plan.world_size, plan.num_params

    def normal(n, scale, dtype):
        out = torch.empty(n, dtype=dtype, device=dev)
        step_n = 1 << 27
        for s in range(0, n, step_n):
            e = min(n, s + step_n)
            out[s:e] = (torch.randn(e - s, generator=gen, device=dev) * scale).to(dtype)
        return out

    if name == "ag_pack":
        shards = [torch.ones(plan.local_elems(p, rank), device=dev) if wl.is_norm[p]
                  else normal(plan.local_elems(p, rank), 0.02, torch.float32) for p in range(P)]
        out = torch.empty(S, dtype=torch.bfloat16, device=dev)
        return (lambda st: plan.ag_pack(rank, shards, out, st)), (shards, out)
    if name == "ag_unpack":
        gathered = normal(W * S, 0.02, torch.bfloat16)
        params = [torch.empty(n * k, dtype=torch.bfloat16, device=dev) for n, k in wl.dims]
        return (lambda st: plan.ag_unpack(gathered, params, st)), (gathered, params)
    if name == "rs_pack":
        grads = [normal(n * k, 1e-3, torch.bfloat16) for n, k in wl.dims]
        send = torch.empty(W * S, dtype=torch.bfloat16, device=dev)
        return (lambda st: plan.rs_pack(grads, send, st)), (grads, send)
    recv = normal(W * S, 1e-3, torch.bfloat16)
    outs = [torch.empty(plan.local_elems(p, rank), dtype=torch.float32, device=dev) for p in range(P)]
    return (lambda st: plan.rs_reduce(rank, recv, outs, st)), (recv, outs)


def time_launches(calls, reps, stream, labels=None, label=None, warm=3):
    """``reps`` launches cycling through ``calls`` (one per input/output set),
    after ``warm`` untimed ones, with the device kept busy by a wait kernel
    while the host enqueues them all: the HIP events then see device time
    only.  Returns the per-launch times (event pairs between consecutive
    launches, ms) and the average over all of them back to back (one pair)."""
    import torch

    n = len(calls)
    for k in range(max(warm, 1)):
        calls[k % n](stream)
        if labels is not None:
            labels.append(label)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    with torch.cuda.stream(stream):
        torch.cuda._sleep(SLEEP_CYCLES)
    ev[0].record(stream)
    for k in range(reps):
        calls[k % n](stream)
        ev[k + 1].record(stream)
        if labels is not None:
            labels.append(label)
    torch.cuda.synchronize()
    per = [ev[k].elapsed_time(ev[k + 1]) for k in range(reps)]
    return per, ev[0].elapsed_time(ev[reps]) / reps


def kernel_leg(plan, wl, rank, reps, dev, stream, labels=None, kernels=KERNELS, tag=""):
    """Each of ``kernels`` ``reps`` times over rotating input/output sets of
    more than ROTATE_BYTES in total; per kernel: event statistics.  Launches
    are labelled name + tag."""
    import torch

    W, S, E = plan.world_size, plan.chunk_elems, wl.total_elems
    V0 = sum(plan.local_elems(p, rank) for p in range(plan.num_params))
    abytes = algorithmic_bytes(W, S, E, V0)
    gen = torch.Generator(device=dev)
    gen.manual_seed(2000 + wl.key)
    res = {}
    for name in kernels:
        nsets = min(64, max(2, -(-ROTATE_BYTES // abytes[name])))
        sets = [kernel_set(name, plan, wl, rank, dev, gen) for _ in range(nsets)]
        torch.cuda.synchronize()
        per, b2b = time_launches([c for c, _ in sets], reps, stream, labels, name + tag, warm=min(nsets, 8))
        res[name] = {"reps": reps, "sets": nsets, "set_bytes": abytes[name], **{
            "event_" + k: v for k, v in stats_us(per).items()}, "b2b_avg_us": round(b2b * 1e3, 3)}
        del sets
        torch.cuda.empty_cache()
    return res


# ----------------------------------------------------------------- ceilings: reference streams

CEILINGS = ("probe_read", "probe_fill", "probe_copy", "probe_cast", "probe_reduce_store", "probe_reduce_nostore")


def load_probes():
    """The reference-stream library (built beside the bucket library)."""
    import ctypes

    import torch  # noqa: F401  (the probes bind to torch's HIP runtime)

    if not os.path.exists(PROBES_LIB):
        raise ImportError(f"{PROBES_LIB} is not built: run `python -m paper_2411_00284_amd.build`")
    lib = ctypes.CDLL(PROBES_LIB)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
    sigs = {"probe_read": [vp, i64, vp, vp], "probe_fill": [vp, i64, vp], "probe_copy": [vp, vp, i64, vp],
            "probe_cast": [vp, vp, i64, vp], "probe_strided_reduce": [vp, i64, i32, vp, i64, i32, vp, vp],
            "probe_empty": [i64, i32, vp]}
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    return lib


def ceiling_bytes(plan, rank):
    """Bytes each reference stream moves at the bucket's shapes: the W*S
    buffer read, filled and copied; the rank's fp32 shard elements cast; the
    rank's outputs (whole 4096-element tiles) reduced over W strided sources,
    with and without storing them."""
    W, S = plan.world_size, plan.chunk_elems
    V0 = sum(plan.local_elems(p, rank) for p in range(plan.num_params))
    n4 = V0 // 4
    nr = V0 // 4096 * 4096
    return {"probe_read": 2 * W * S, "probe_fill": 2 * W * S, "probe_copy": 4 * W * S, "probe_cast": 24 * n4,
            "probe_reduce_store": 2 * W * nr + 4 * nr, "probe_reduce_nostore": 2 * W * nr}


def ceiling_set(name, plan, rank, dev, gen, lib, sink):
    """One input/output set of a reference stream; returns its call and tensors."""
    import torch

    W, S = plan.world_size, plan.chunk_elems
    V0 = sum(plan.local_elems(p, rank) for p in range(plan.num_params))

    def check(rc):
        if rc != 0:
            raise RuntimeError(f"{name}: HIP error {rc}")

    if name in ("probe_read", "probe_fill", "probe_copy"):
        src = torch.randn(W * S, generator=gen, device=dev).to(torch.bfloat16)
        n16 = W * S * 2 // 16
        if name == "probe_read":
            return (lambda st: check(lib.probe_read(src.data_ptr(), n16, sink.data_ptr(), st.cuda_stream))), (src,)
        if name == "probe_fill":
            return (lambda st: check(lib.probe_fill(src.data_ptr(), n16, st.cuda_stream))), (src,)
        dst = torch.empty_like(src)
        return (lambda st: check(lib.probe_copy(src.data_ptr(), dst.data_ptr(), n16, st.cuda_stream))), (src, dst)
    if name == "probe_cast":
        n4 = V0 // 4
        src = torch.randn(4 * n4, generator=gen, device=dev) * 0.02
        dst = torch.empty(4 * n4, dtype=torch.bfloat16, device=dev)
        return (lambda st: check(lib.probe_cast(src.data_ptr(), dst.data_ptr(), n4, st.cuda_stream))), (src, dst)
    nr = V0 // 4096 * 4096
    store = 1 if name == "probe_reduce_store" else 0
    src = (torch.randn(W * S, generator=gen, device=dev) * 1e-3).to(torch.bfloat16)
    dst = torch.empty(max(nr, 4), dtype=torch.float32, device=dev)
    return (lambda st: check(lib.probe_strided_reduce(src.data_ptr(), S, W, dst.data_ptr(), nr, store,
                                                       sink.data_ptr(), st.cuda_stream))), (src, dst)


def ceiling_leg(plan, rank, reps, dev, stream, labels=None):
    """Each reference stream ``reps`` times over rotating sets, as the
    per-kernel leg times the library's calls."""
    import torch

    lib = load_probes()
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(4000)
    nbytes = ceiling_bytes(plan, rank)
    res = {}
    for name in CEILINGS:
        if nbytes[name] == 0:
            continue
        nsets = min(64, max(2, -(-ROTATE_BYTES // nbytes[name])))
        sets = [ceiling_set(name, plan, rank, dev, gen, lib, sink) for _ in range(nsets)]
        torch.cuda.synchronize()
        per, b2b = time_launches([c for c, _ in sets], reps, stream, labels, name, warm=min(nsets, 8))
        res[name] = {"bytes": nbytes[name], "sets": nsets, **{"event_" + k: v for k, v in stats_us(per).items()},
                     "b2b_avg_us": round(b2b * 1e3, 3)}
        del sets
        torch.cuda.empty_cache()
    return res


# ----------------------------------------------------------------- kernel trace of a child run

def short_symbol(name):
    """A trace's kernel name without return type, namespaces or parameter list."""
    name = name.replace("(anonymous namespace)::", "").replace("fsdp::", "")
    if name.startswith("void "):
        name = name[5:]
    depth = 0
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return name[:i].strip()
    return name.strip()


def rocprof_path():
    import shutil
    return shutil.which("rocprofv3") or ("/opt/rocm/bin/rocprofv3" if os.path.exists("/opt/rocm/bin/rocprofv3")
                                         else None)


def progress(msg):
    """A progress line on stderr (the JSON line alone goes to stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def traced_child(spec, timeout=300):
    spec = dict(spec)
    from paper_2411_00284_amd import _native
    if os.path.abspath(_native.LIB_PATH) != os.path.abspath(os.path.join(ROOT, "paper_2411_00284_amd",
                                                                         "libfsdp_bucket.so")):
        spec["library"] = _native.LIB_PATH
    return _traced_child(spec, timeout)


def _traced_child(spec, timeout):
    """Run ``bench.py --child`` with ``spec`` as a child process under
    ``rocprofv3 --kernel-trace`` and return (child result, per-launch kernel
    durations in ms grouped by the child's labels, kernel names per label), or
    (None, None, reason).  The child labels every library launch it makes, in
    order; the trace's dispatches of the library kernels are matched to them
    one to one."""
    import csv
    import glob
    import shutil
    import subprocess
    import tempfile

    prof = rocprof_path()
    if prof is None:
        return None, None, "rocprofv3 not found"
    tmp = tempfile.mkdtemp(prefix="bench_trace_")
    try:
        spec_path = os.path.join(tmp, "spec.json")
        out_path = os.path.join(tmp, "child.json")
        with open(spec_path, "w") as f:
            json.dump(spec, f)
        cmd = [prof, "--kernel-trace", "-f", "csv", "-d", os.path.join(tmp, "trace"), "-o", "trace", "--",
               sys.executable, os.path.abspath(__file__), "--child", spec_path, out_path]
        env = dict(os.environ, TMPDIR=tmp)
        try:
            res = subprocess.run(cmd, cwd=tmp, env=env, capture_output=True, text=True, timeout=timeout)
        except subprocess.TimeoutExpired:
            return None, None, "traced child run timed out"
        csvs = glob.glob(os.path.join(tmp, "trace", "**", "*kernel_trace.csv"), recursive=True)
        if not os.path.exists(out_path) or not csvs:
            return None, None, f"traced child run failed (rc {res.returncode}): {res.stderr[-400:]}"
        child = json.load(open(out_path))
        rows = []
        with open(csvs[0]) as f:
            for r in csv.DictReader(f):
                name = r["Kernel_Name"]
                if any(b in name for b in KERNEL_BASENAMES):
                    key = int(r.get("Dispatch_Id") or 0), int(r["Start_Timestamp"])
                    rows.append((key, (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-6, name))
        rows.sort()
        labels = child["labels"]
        if len(rows) != len(labels):
            return None, None, f"{len(rows)} library dispatches traced for {len(labels)} launches"
        per, names = {}, {}
        for (_, ms, name), lab in zip(rows, labels):
            per.setdefault(lab, []).append(ms)
            names.setdefault(lab, short_symbol(name))
        return child, per, names
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


def use_library(path):
    """Point the binding at another build of the library (before it loads)."""
    from paper_2411_00284_amd import _native

    if _native._lib is not None:
        raise RuntimeError("the library is already loaded")
    _native.LIB_PATH = os.path.abspath(path)


def child_main(spec_path, out_path):
    """The traced child: runs the leg the spec names and writes its labels."""
    import torch

    spec = json.load(open(spec_path))
    if spec.get("library"):
        use_library(spec["library"])

    from paper_2411_00284_amd import BucketPlan
    from synth import workload

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    labels = []
    out = {"spec": spec}
    if spec["mode"] == "kernels":
        wl = workload(spec["workload"])
        plan = BucketPlan(wl.world_size, wl.dims, spec.get("align", 8))
        out["events"] = kernel_leg(plan, wl, spec["rank"], spec["reps"], dev, stream, labels)
        if spec.get("ceilings"):
            out["ceilings"] = ceiling_leg(plan, spec["rank"], spec["reps"], dev, stream, labels)
        plan.close()
    elif spec["mode"] == "records":
        wl = workload(spec["workload"])
        plan = BucketPlan(wl.world_size, wl.dims)
        for r in spec["ranks"]:
            kernel_leg(plan, wl, r, spec["reps"], dev, stream, labels, record_kernels(r), f"@{r}")
        plan.close()
    elif spec["mode"] == "pack_sweep":
        out["cases"] = pack_sweep_leg(spec["reps"], dev, stream, labels)
        out["empty"] = empty_launch_leg(spec["reps"], stream, labels)
    out["labels"] = labels
    with open(out_path, "w") as f:
        json.dump(out, f)
    return 0


# ----------------------------------------------------------------- result records

RECORD_WORKLOADS = (1, 2, 3, 4, 5, 6, 7)


def record_kernels(rank):
    """The calls recorded at a rank: all four at rank 0; at the other ranks
    the two whose work depends on the rank (the unpack and rs_pack read and
    write the whole block at every rank)."""
    return KERNELS if rank == 0 else ("ag_pack", "rs_reduce")


def oracle_inputs(name, wl, plan, rank):
    """The oracle's inputs of one call (random bit patterns, finite where the
    call computes with them), as the CPU-baseline leg draws them."""
    import numpy as np

    import oracle.fsdp_oracle as O
    from synth import random_bits16, random_bits32

    W, S = plan.world_size, plan.chunk
    if name == "ag_pack":
        shards = [random_bits32([1, p], O.local_elems(plan, p, rank)).view(np.float32) for p in range(len(wl.dims))]
        return [np.where(np.isfinite(s), s, np.float32(0)) for s in shards]
    if name == "ag_unpack":
        return random_bits16([2], W * S)
    if name == "rs_pack":
        return [random_bits16([3, p], n * k).reshape(n, k) for p, (n, k) in enumerate(wl.dims)]
    return random_bits16([4], W * S) & np.uint16(0xBFFF)


def oracle_call(name, plan, rank, x):
    import oracle.fsdp_oracle as O

    if name == "ag_pack":
        return O.ag_pack(plan, rank, x)
    if name == "ag_unpack":
        return O.ag_unpack(plan, x)
    if name == "rs_pack":
        return O.rs_pack(plan, x)
    return O.rs_reduce(plan, rank, x)


def library_matches(name, gpu_plan, rank, x, want):
    """One library call on the oracle's inputs: is every output bit equal?"""
    import numpy as np
    import torch

    dev = torch.device("cuda:0")

    def up16(a):
        return torch.from_numpy(np.ascontiguousarray(a).reshape(-1).view(np.int16)).to(dev).view(torch.bfloat16)

    def down(t, dtype):
        return t.view(torch.int16 if dtype == np.uint16 else torch.int32).cpu().numpy().view(dtype)

    P, S, W = gpu_plan.num_params, gpu_plan.chunk_elems, gpu_plan.world_size
    if name == "ag_pack":
        shards = [torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in x]
        out = torch.empty(S, dtype=torch.bfloat16, device=dev)
        gpu_plan.ag_pack(rank, shards, out)
        ok = bool(np.array_equal(down(out, np.uint16), want))
    elif name == "ag_unpack":
        params = [torch.empty(gpu_plan.full_elems(p), dtype=torch.bfloat16, device=dev) for p in range(P)]
        gpu_plan.ag_unpack(up16(x), params)
        ok = all(np.array_equal(down(params[p], np.uint16), want[p].reshape(-1)) for p in range(P))
    elif name == "rs_pack":
        send = torch.empty(W * S, dtype=torch.bfloat16, device=dev)
        gpu_plan.rs_pack([up16(g) for g in x], send)
        ok = bool(np.array_equal(down(send, np.uint16), want))
    else:
        outs = [torch.empty(gpu_plan.local_elems(p, rank), dtype=torch.float32, device=dev) for p in range(P)]
        gpu_plan.rs_reduce(rank, up16(x), outs)
        ok = all(np.array_equal(down(outs[p], np.uint32), want[p].reshape(-1).view(np.uint32)) for p in range(P))
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return ok


def records_main(out_dir, reps, keys=RECORD_WORKLOADS):
    """One record per (workload, kernel, rank): kernel-trace and event
    statistics of the per-kernel leg, GB/s and share of peak, committed
    counter bytes where they match the source, the oracle's time for the
    same call on the host, and whether the library's output equals the
    oracle's bit for bit on the oracle's inputs (full size)."""
    import torch

    import oracle.fsdp_oracle as O
    from paper_2411_00284_amd import BucketPlan
    from synth import workload

    os.makedirs(out_dir, exist_ok=True)
    cores = len(os.sched_getaffinity(0))
    records = []
    for key in keys:
        wl = workload(key)
        W = wl.world_size
        ranks = sorted({0, W // 2, W - 1})
        print(f"[records] {wl.name}: traced leg", file=sys.stderr, flush=True)
        child, per, names = traced_child({"mode": "records", "workload": key, "ranks": ranks, "reps": reps})
        dev = torch.device("cuda:0")
        torch.cuda.set_device(dev)
        stream = torch.cuda.current_stream()
        plan = BucketPlan(W, wl.dims)
        oplan = O.make_plan(W, wl.dims, 8)
        S, E = plan.chunk_elems, wl.total_elems
        for r in ranks:
            print(f"[records] {wl.name}: rank {r}", file=sys.stderr, flush=True)
            leg = kernel_leg(plan, wl, r, reps, dev, stream, kernels=record_kernels(r))
            V = sum(plan.local_elems(p, r) for p in range(plan.num_params))
            abytes = algorithmic_bytes(W, S, E, V)
            for name in record_kernels(r):
                x = oracle_inputs(name, wl, oplan, r)
                t0 = time.perf_counter()
                want = oracle_call(name, oplan, r, x)
                oracle_s = time.perf_counter() - t0
                parity = library_matches(name, plan, r, x, want)
                del x, want
                lab = f"{name}@{r}"
                tr = stats_us(per[lab][-reps:]) if child is not None and lab in per else None
                us = tr["median_us"] if tr else leg[name]["event_median_us"]
                traffic = read_traffic(name, wl.name) if r == 0 else None
                records.append({
                    "workload": wl.name, "config": key, "world_size": W, "rank": r if name in ("ag_pack", "rs_reduce") else None,
                    "kernel": name, "symbol": names[lab] if tr else kernel_symbol(name, plan, r, cus_of(dev)),
                    "bytes": abytes[name], "reps": reps, "sets": leg[name]["sets"],
                    "event_median_us": leg[name]["event_median_us"], "event_min_us": leg[name]["event_min_us"],
                    "rocprof_median_us": tr["median_us"] if tr else None, "rocprof_min_us": tr["min_us"] if tr else None,
                    "GBps": round(abytes[name] / (us * 1e-6) / 1e9, 1),
                    "frac": round(abytes[name] / (us * 1e-6) / 1e9 / PEAK_GBPS, 4),
                    "counter_bytes": traffic, "counter_ratio": None if traffic is None else round(traffic / abytes[name], 4),
                    "oracle_s": round(oracle_s, 3), "oracle_threads": 1, "host_cores": cores,
                    "oracle_GBps": round(abytes[name] / oracle_s / 1e9, 3), "parity": parity,
                    "kernel_source_sha256": kernel_source_sha(),
                })
        plan.close()
        torch.cuda.empty_cache()
    with open(os.path.join(out_dir, "records.jsonl"), "w") as f:
        for rec in records:
            f.write(json.dumps(rec) + "\n")
    with open(os.path.join(out_dir, "records.md"), "w") as f:
        f.write(records_table(records))
    print(json.dumps({"records": len(records), "dir": out_dir,
                      "parity": all(r["parity"] for r in records)}), flush=True)
    return 0 if all(r["parity"] for r in records) else 1


def cus_of(dev):
    import torch
    return torch.cuda.get_device_properties(dev).multi_processor_count


def records_table(records):
    lines = ["| workload | W | rank | kernel | algorithmic bytes | trace median us | trace min us | GB/s | % of peak "
             "| event median us | counter / alg | oracle s (1 thread) | bit-exact |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in records:
        lines.append("| {workload} | {world_size} | {rk} | {kernel} | {bytes} | {tm} | {tn} | {GBps} | {pct:.1f} | "
                     "{event_median_us} | {cr} | {oracle_s} | {par} |".format(
                         **r, rk="all" if r["rank"] is None else r["rank"], tm=r["rocprof_median_us"],
                         tn=r["rocprof_min_us"], pct=100 * r["frac"],
                         cr="" if r["counter_ratio"] is None else r["counter_ratio"],
                         par="yes" if r["parity"] else "NO"))
    return "\n".join(lines) + "\n"


# ----------------------------------------------------------------- ag_pack over bucket sizes

def pack_sweep_cases():
    """Buckets for the pack's size sweep: one Llama-3 block (8B, 70B, 405B
    shapes) at several world sizes, so one rank's chunk spans 10 to 320 MB of
    algorithmic bytes, plus one-parameter buckets of 1, 64 and 512 tiles for
    the fixed cost of a launch."""
    from synth.workloads import KV_ROWS, Workload, _block

    blocks = {"8b": (4096, 14336), "70b": (8192, 28672), "405b": (16384, 53248)}
    cases = [Workload(0, f"one-param-{t}-tiles", 1, ("x",), ((t * 1024, 1),), (False,)) for t in (1, 64, 512)]
    for blk, w in (("8b", 128), ("8b", 64), ("70b", 128), ("8b", 32), ("70b", 64), ("8b", 16), ("405b", 128),
                   ("70b", 32), ("8b", 8), ("405b", 64), ("70b", 16)):
        d, f = blocks[blk]
        cases.append(_block(0, f"llama3-{blk}-block-w{w}", w, d, f, KV_ROWS))
    return cases


def pack_sweep_leg(reps, dev, stream, labels):
    import torch

    from paper_2411_00284_amd import BucketPlan

    gen = torch.Generator(device=dev)
    gen.manual_seed(3000)
    res = []
    for wl in pack_sweep_cases():
        plan = BucketPlan(wl.world_size, wl.dims)
        S = plan.chunk_elems
        V0 = sum(plan.local_elems(p, 0) for p in range(wl.num_params))
        nbytes = 4 * V0 + 2 * S
        nsets = min(200, max(2, -(-ROTATE_BYTES // nbytes)))
        sets = [kernel_set("ag_pack", plan, wl, 0, dev, gen) for _ in range(nsets)]
        torch.cuda.synchronize()
        per, b2b = time_launches([c for c, _ in sets], reps, stream, labels, wl.name, warm=min(nsets, 8))
        res.append({"name": wl.name, "world_size": wl.world_size, "bytes": nbytes, "sets": nsets,
                    **{"event_" + k: v for k, v in stats_us(per).items()}, "b2b_avg_us": round(b2b * 1e3, 3)})
        del sets
        plan.close()
        torch.cuda.empty_cache()
    return res


def pack_tiles(plan, tile):
    """Work tiles of the single-chunk pack with tiles of ``tile`` elements."""
    ends = [plan.offset(p + 1) for p in range(plan.num_params - 1)] + [plan.chunk_elems]
    return sum(-(-(e - plan.offset(p)) // tile) for p, e in enumerate(ends))


def empty_launch_cases():
    """Grids that move nothing, for the part of a launch's fixed cost that is
    dispatch and retirement: one small-tile workgroup, and the 70B block's
    pack grid (W = 64) in its big and small tiles."""
    from paper_2411_00284_amd import BucketPlan
    from synth import workload

    wl = workload(3)
    plan = BucketPlan(wl.world_size, wl.dims)
    big, small = pack_tiles(plan, PACK_BIG_TILE), pack_tiles(plan, PACK_SMALL_TILE)
    plan.close()
    return [("empty-1x128", 1, 128), (f"empty-{big}x256", big, 256), (f"empty-{small}x128", small, 128)]


def empty_launch_leg(reps, stream, labels):
    lib = load_probes()
    res = []
    for name, grid, threads in empty_launch_cases():
        def call(st, grid=grid, threads=threads):
            rc = lib.probe_empty(grid, threads, st.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"probe_empty: HIP error {rc}")
        per, b2b = time_launches([call, call], reps, stream, labels, name, warm=2)
        res.append({"name": name, "grid": grid, "threads": threads,
                    **{"event_" + k: v for k, v in stats_us(per).items()}, "b2b_avg_us": round(b2b * 1e3, 3)})
    return res


def pack_sweep(reps):
    """The pack over pack_sweep_cases(), timed by a live kernel trace; fits
    T = t0 + bytes / BW to the trace medians of the block buckets and reports
    the one-parameter buckets' median as the launch floor."""
    import numpy as np

    child, per, names = traced_child({"mode": "pack_sweep", "reps": reps})
    if child is None:
        return {"error": names}
    rows = []
    for c in child["cases"]:
        d = per[c["name"]][-reps:]
        st = stats_us(d)
        rows.append({**c, **{"rocprof_" + k: v for k, v in st.items()},
                     "GBps_rocprof_median": round(c["bytes"] / (st["median_us"] * 1e-6) / 1e9, 1)})
    blocks = [r for r in rows if r["name"].startswith("llama3")]
    x = np.array([r["bytes"] for r in blocks], dtype=np.float64)
    y = np.array([r["rocprof_median_us"] for r in blocks], dtype=np.float64)
    beta, t0 = np.polyfit(x, y, 1)
    r2 = 1.0 - float(np.sum((y - (t0 + beta * x)) ** 2) / np.sum((y - y.mean()) ** 2))
    floor = float(np.median([r["rocprof_median_us"] for r in rows if r["name"].startswith("one-param")]))
    empty = []
    for c in child.get("empty", []):
        st = stats_us(per[c["name"]][-reps:])
        empty.append({**c, **{"rocprof_" + k: v for k, v in st.items()}})
    return {"kernel": names.get(blocks[0]["name"]), "reps": reps, "cases": rows,
            "fit": {"t0_us": round(float(t0), 3), "GBps": round(1e-3 / float(beta), 1), "r2": round(r2, 5),
                    "points": len(blocks)},
            "launch_floor_us": round(floor, 3), "empty_launches": empty}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, help="1 toy, 2 8B, 3 70B (default), 4 405B, 5 uneven, 6 70B TP-8 shards, 7 8B at W=128")
    ap.add_argument("--rank", type=int, default=0, help="the rank whose share is timed (0 <= rank < W)")
    ap.add_argument("--align", type=int, default=8,
                    help="the plan's alignment A in elements (8: 16-byte segments; 1: the dense concatenation)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip timing the fp32-wire and chunk-table forms after the steps")
    ap.add_argument("--variant-reps", type=int, default=10)
    ap.add_argument("--event-every", type=int, default=5,
                    help="record the per-kernel HIP events on every N-th timed step (N=1: every step)")
    ap.add_argument("--kernel-reps", type=int, default=30,
                    help="launches per kernel in the per-kernel leg (rotating sets, device kept ahead)")
    ap.add_argument("--no-trace", action="store_true",
                    help="skip the per-kernel leg's rocprofv3 kernel trace (a child run)")
    ap.add_argument("--ceilings", action="store_true",
                    help="also time reference streams (read, fill, copy, cast, strided reduce) at the bucket's shapes")
    ap.add_argument("--pack-sweep", action="store_true",
                    help="also time ag_pack over buckets of 10-320 MB by kernel trace and fit t0 + bytes/BW")
    ap.add_argument("--copy-cost", action="store_true",
                    help="also fit the alpha + beta*bytes copy cost over sub-buckets of the block "
                         "(launches the path kernels at other sizes, so it is off in profiled runs)")
    ap.add_argument("--graph", action="store_true",
                    help="also time the step replayed from a HIP graph")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after the steps, run a plain 1 GiB device copy (for counter scaling)")
    ap.add_argument("--records", metavar="DIR",
                    help="instead of the steps: one record per (workload, kernel, rank) for workloads 1-7, "
                         "written to DIR/records.jsonl and DIR/records.md")
    ap.add_argument("--record-workloads", type=int, nargs="+", default=list(RECORD_WORKLOADS),
                    help="the workloads --records covers (default: all seven)")
    ap.add_argument("--library", metavar="SO",
                    help="load this build of libfsdp_bucket.so (a launch-shape variant made with "
                         "`python -m paper_2411_00284_amd.build -DNAME=VALUE --out DIR`) instead of the package's")
    ap.add_argument("--child", nargs=2, metavar=("SPEC", "OUT"), help=argparse.SUPPRESS)
    args = ap.parse_args(argv)

    if args.library:
        use_library(args.library)
    if args.child:
        return child_main(*args.child)
    if args.records:
        return records_main(args.records, max(1, args.kernel_reps), tuple(args.record_workloads))
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

    reps = max(1, args.kernel_reps)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    plan = BucketPlan(W, wl.dims, args.align)
    S = plan.chunk_elems
    P = wl.num_params
    E = wl.total_elems
    V0 = sum(plan.local_elems(p, rank) for p in range(P))
    stream = torch.cuda.current_stream()

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

    progress(f"{wl.name}: {args.warmup} warm-up and {args.steps} timed steps")
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

    # ---- the per-kernel leg, after the steps (so that neither its allocations
    # nor its seconds of streaming precede the timed steps): each call over
    # rotating sets of > 1.5 GiB, here by HIP events and in a child process
    # under a kernel trace
    progress("per-kernel leg (HIP events)")
    leg = kernel_leg(plan, wl, rank, reps, dev, stream)
    trace = None
    if not args.no_trace:
        progress("per-kernel leg under a rocprofv3 kernel trace (child process)")
        child, per, names = traced_child({"mode": "kernels", "workload": args.workload, "rank": rank, "reps": reps,
                                          "ceilings": args.ceilings, "align": args.align})
        trace = {"error": names} if child is None else {
            name: {"symbol": names[name], **{"rocprof_" + k: v for k, v in stats_us(per[name][-reps:]).items()}}
            for name in per}
    ceilings = None
    if args.ceilings:
        ceilings = ceiling_leg(plan, rank, reps, dev, stream)
        for name, c in ceilings.items():
            tr = trace.get(name) if trace and "error" not in trace else None
            us = tr["rocprof_median_us"] if tr else c["event_median_us"]
            c["trace"] = tr
            c["GBps"] = round(c["bytes"] / (us * 1e-6) / 1e9, 1)
            c["frac"] = round(c["bytes"] / (us * 1e-6) / 1e9 / PEAK_GBPS, 4)

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
        lg = leg[name]
        tr = trace.get(name) if trace and "error" not in trace else None
        kernel_us = tr["rocprof_median_us"] if tr else lg["event_median_us"]
        gbps = abytes[name] / (kernel_us * 1e-6) / 1e9
        kernels[name] = {
            "symbol": tr["symbol"] if tr else kernel_symbol(name, plan, rank, cus),
            "bytes": abytes[name],
            "GBps": round(gbps, 1), "frac": round(gbps / PEAK_GBPS, 4),
            "timing": "rocprofv3 kernel trace median (live)" if tr else "HIP event median",
            "leg": lg,
            "leg_frac_event_median": round(abytes[name] / (lg["event_median_us"] * 1e-6) / 1e9 / PEAK_GBPS, 4),
            "trace": tr,
            "step_event_avg_us": round(avg_ms * 1e3, 2),
            "step_event_median_us": round(float(np.median(per_kernel_ms[name])) * 1e3, 2),
            "step_event_samples": len(per_kernel_ms[name]),
            "committed_rocprof_avg_us": read_profile_avg_us(name, wl.name),
        }

    copy_ref = None if args.no_variants else time_d2d_copy(gathered, send_buf, stream, args.variant_reps)

    # (the chunk-table forms need 16-byte-aligned chunks: a dense bucket with an
    # odd chunk stride skips them)
    variants = None if args.no_variants or (2 * S) % 16 else time_variants(
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

    # The roofline entry: the kernel with the longest launches in the timed
    # steps, at its HIP-event average over those steps.
    dominant = max(KERNELS, key=lambda n: kernels[n]["step_event_avg_us"])
    dom = kernels[dominant]
    dom_gbps = abytes[dominant] / (dom["step_event_avg_us"] * 1e-6) / 1e9
    roofline = {
        "bound": "hbm",
        "kernel": dom["symbol"],
        "achieved": round(dom_gbps, 1),
        "peak": PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(dom_gbps / PEAK_GBPS, 4),
        "traffic": read_traffic(dominant, wl.name),
    }

    cpu = None
    if not args.no_cpu_baseline:
        progress("CPU oracle baseline and full-size parity")
        cpu = cpu_baseline(wl, rank, gpu_plan=plan, align=args.align)

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
                   "block_elems": E, "rank_elems": V0, "align_elems": args.align, "wire": "bf16",
                   "step": "ag_pack+ag_unpack+rs_pack+rs_reduce", "step_bytes": step_bytes},
        "frac_of_peak": round(step_bytes / (elapsed / args.steps) / 1e9 / PEAK_GBPS, 4),
        "kernels": kernels,
        "kernel_trace": trace.get("error") if trace and "error" in trace else (
            None if trace is None else "rocprofv3 --kernel-trace of the per-kernel leg in a child process"),
        "roofline": roofline,
        "d2d_copy": copy_ref,
        "cpu_baseline": cpu,
        "variants": variants,
        "auto_wrap": None if args.no_variants else time_auto_wrap(wl),
        "copy_cost": fit_copy_cost(wl, stream) if args.copy_cost else None,
        "graph": None if not args.graph else time_graph_step(
            lambda: run_step(None, torch.cuda.current_stream()), args.steps),
        "ceilings": ceilings,
        "pack_sweep": pack_sweep(reps) if args.pack_sweep else None,
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


def cpu_baseline(wl, rank=0, min_seconds=10.0, max_passes=50, gpu_plan=None, align=8):
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
    plan = O.make_plan(W, dims, align)
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
