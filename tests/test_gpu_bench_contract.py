"""The benchmark's one JSON line, from a short run on the toy block: the
fields a reader of the line relies on are present and consistent."""

from __future__ import annotations

import json
import os
import subprocess
import sys

import pytest
import torch

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line_on_the_toy_block():
    print("bench.py --workload 1 --steps 3 --warmup 1", flush=True)
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "1", "--steps", "3",
                          "--warmup", "1", "--variant-reps", "1", "--event-every", "1"],
                         capture_output=True, text=True, timeout=240)
    assert res.returncode == 0, res.stderr[-2000:]
    lines = [l for l in res.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline", "kernels"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1 and d["higher_is_better"] is True
    assert d["config"]["workload"] == "toy-block-w4" and d["config"]["world_size"] == 4
    step_bytes = sum(k["bytes"] for k in d["kernels"].values())
    assert step_bytes == d["config"]["step_bytes"]
    assert d["value"] > 0 and abs(d["value"] - step_bytes / (d["ms_per_step"] * 1e-3) / 1e9) < 0.01 * d["value"] + 0.2
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-3
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["cores"] == 1 and cpu["value"] > 0
    # the library on the oracle's own inputs, compared bit for bit inside the bench
    assert cpu["parity"] == {"ag_pack": True, "ag_unpack": True, "rs_pack": True, "rs_reduce": True}
    assert set(d["kernels"]) == {"ag_pack", "ag_unpack", "rs_pack", "rs_reduce"}
    # the per-kernel leg: >= 30 launches per kernel over rotating sets of more
    # than 1.5 GiB (or the 64-set cap), timed by events and by a kernel trace
    for name, k in d["kernels"].items():
        leg = k["leg"]
        assert leg["reps"] >= 30 and leg["sets"] >= 2
        assert leg["sets"] * leg["set_bytes"] > 3 << 29 or leg["sets"] == 64
        assert 0 < leg["event_min_us"] <= leg["event_median_us"]
        assert k["symbol"].startswith(name + "_kernel<"), k["symbol"]
        if k["trace"] is not None:
            assert 0 < k["trace"]["rocprof_min_us"] <= k["trace"]["rocprof_median_us"]
            assert k["timing"].startswith("rocprofv3")
    assert d["kernel_trace"] is not None
    assert d["d2d_copy"]["bytes"] == 2 * 2 * 4 * d["config"]["chunk_elems"]


def test_records_on_the_toy_block(tmp_path):
    """--records: one record per (workload, kernel, rank), every one bit-exact
    against the oracle and carrying the per-kernel leg's statistics."""
    print("bench.py --records (toy block)", flush=True)
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--records", str(tmp_path),
                          "--record-workloads", "1"], capture_output=True, text=True, timeout=240)
    assert res.returncode == 0, res.stderr[-2000:]
    recs = [json.loads(l) for l in open(tmp_path / "records.jsonl")]
    # ranks 0, 2 and 3 of W = 4: four calls at rank 0, the two per-rank calls at the others
    assert len(recs) == 8
    assert sorted((r["kernel"], r["rank"]) for r in recs) == sorted(
        [("ag_pack", 0), ("ag_pack", 2), ("ag_pack", 3), ("rs_reduce", 0), ("rs_reduce", 2), ("rs_reduce", 3),
         ("ag_unpack", None), ("rs_pack", None)])
    for r in recs:
        assert r["parity"] is True and r["reps"] >= 30 and r["bytes"] > 0
        assert r["rocprof_median_us"] is None or r["rocprof_median_us"] > 0
        assert 0 < r["frac"] and r["oracle_threads"] == 1
    assert (tmp_path / "records.md").read_text().count("| yes |") == 8
