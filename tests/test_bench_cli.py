"""Host-side checks of the benchmark's command line and its CPU baseline leg
(no GPU is touched: both refusals return before the device is selected)."""

import bench
from synth import workload


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU only" in capsys.readouterr().err


def test_rank_outside_world_is_refused(capsys):
    assert bench.main(["--workload", "1", "--rank", "4"]) == 2      # the toy block has W = 4
    assert "outside 0..3" in capsys.readouterr().err
    assert bench.main(["--workload", "1", "--rank", "-1"]) == 2


def test_cpu_baseline_at_another_rank():
    wl = workload(1)
    res = bench.cpu_baseline(wl, rank=3, min_seconds=0.0, max_passes=1)
    assert res["kind"] == "oracle" and res["cores"] == 1 and res["value"] > 0
    assert "rank 3" in res["sample"]
    assert set(res["per_pass_s"]) == set(bench.KERNELS)


def test_algorithmic_bytes_of_the_70b_block():
    # the per-kernel byte counts of the 70B block at rank 0 (W = 64, S = V_0 = 13,369,600)
    b = bench.algorithmic_bytes(64, 13369600, 855654400, 13369600)
    assert b == {"ag_pack": 80217600, "ag_unpack": 3422617600, "rs_pack": 3422617600, "rs_reduce": 1764787200}


def test_short_symbol_strips_namespaces_and_parameters():
    long = ("void fsdp::(anonymous namespace)::rs_reduce_kernel<fsdp::(anonymous namespace)::ContigChunks, "
            "unsigned short, 256, false>(fsdp::(anonymous namespace)::ReduceArgs<fsdp::(anonymous namespace)::"
            "ContigChunks>)")
    assert bench.short_symbol(long) == "rs_reduce_kernel<ContigChunks, unsigned short, 256, false>"
    assert bench.short_symbol("(anonymous namespace)::probe_copy_kernel(unsigned int __vector(4) const*, long)") \
        == "probe_copy_kernel"


def test_kernel_symbols_follow_the_library_choices():
    """The symbol each call launches: the pack's tile by bucket size, the
    reduce's tile by shard size, the off-grid forms for buckets that need them
    (the host-side rules, checked on the planner's own plans)."""
    from paper_2411_00284_amd import BucketPlan

    def syms(key, align=8, cus=256):
        wl = workload(key)
        plan = BucketPlan(wl.world_size, wl.dims, align)
        out = {n: bench.kernel_symbol(n, plan, 0, cus) for n in bench.KERNELS}
        plan.close()
        return out

    s70 = syms(3)
    assert s70 == bench.KERNEL_SYMBOLS
    toy = syms(1)
    assert toy["ag_pack"] == bench.PACK_SMALL_SYMBOL and toy["rs_reduce"] == bench.REDUCE_SMALL_SYMBOL
    uneven = syms(5)
    assert uneven["ag_unpack"].endswith("true>") and uneven["rs_pack"].endswith("true>")
    assert uneven["rs_reduce"].endswith("false>")          # every offset is on the grid at align 8
    dense = syms(5, align=1)
    assert all(dense[n].endswith("true>") for n in ("ag_unpack", "rs_pack", "rs_reduce"))
    assert syms(2, align=1) == syms(2)                      # every L_p of a Llama block is a multiple of 8


def test_stats_and_records_table():
    st = bench.stats_us([0.002, 0.001, 0.003])
    assert st == {"median_us": 2.0, "min_us": 1.0, "mean_us": 2.0}
    rec = {"workload": "w", "world_size": 4, "rank": None, "kernel": "ag_unpack", "bytes": 10,
           "rocprof_median_us": 1.0, "rocprof_min_us": 0.5, "GBps": 10.0, "frac": 0.00125,
           "event_median_us": 2.0, "counter_ratio": 1.0001, "oracle_s": 0.1, "parity": False}
    table = bench.records_table([rec])
    row = table.strip().splitlines()[-1]
    assert row.startswith("| w | 4 | all | ag_unpack | 10 |") and row.endswith("| 1.0001 | 0.1 | NO |")


def test_pack_sweep_cases_span_the_sizes():
    cases = bench.pack_sweep_cases()
    assert [c.name for c in cases[:3]] == ["one-param-1-tiles", "one-param-64-tiles", "one-param-512-tiles"]
    assert {c.world_size for c in cases[3:]} == {8, 16, 32, 64, 128}


def test_empty_launch_grids_are_the_70b_pack_grids():
    # 13,369,600-element chunk of the 70B block at W = 64 (9 parameters): the
    # big-tile grid is the pack's 8192-element tile count, the small-tile grid
    # its 1024-element tile count, and the big one is what the library launches
    cases = bench.empty_launch_cases()
    assert cases[0] == ("empty-1x128", 1, 128)
    (_, big, tb), (_, small, ts) = cases[1], cases[2]
    assert (tb, ts) == (256, 128)
    assert 13369600 // 8192 <= big <= 13369600 // 8192 + 9
    assert 13369600 // 1024 <= small <= 13369600 // 1024 + 9
    assert big >= bench.PACK_BIG_TILES_PER_CU * 256
