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
