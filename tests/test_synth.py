"""Synthetic workload shapes and seeded generators (no GPU)."""

import numpy as np

from oracle_checks import read_table
from synth import WORKLOADS, grad_rows_bits, param_rows, random_bits16


def test_block_shapes_follow_llama31_table():
    table = {r[0]: (int(r[2]), int(r[3])) for r in read_table("llama31_table2.txt")}
    for key, model in ((2, "8B"), (3, "70B"), (4, "405B"), (7, "8B")):
        dim, ffn = table[model]
        wl = WORKLOADS[key]
        d = dict(zip(wl.names, wl.dims))
        assert d["wq"] == (dim, dim) and d["wo"] == (dim, dim)
        assert d["wk"] == (1024, dim) and d["wv"] == (1024, dim)
        assert d["w1"] == (ffn, dim) and d["w3"] == (ffn, dim) and d["w2"] == (dim, ffn)
        assert d["attention_norm"] == (dim, 1) and d["ffn_norm"] == (dim, 1)
    assert [w.world_size for w in WORKLOADS.values()] == [4, 8, 64, 128, 48, 8, 128]


def test_tp_block_is_one_tp_rank_of_the_70b_block():
    """Workload 6 holds one of 8 tensor-parallel ranks' shards of the 70B block:
    8 of them make up workload 3's parameters (rows split for the column-parallel
    weights, columns for the row-parallel ones, norms whole)."""
    full = dict(zip(WORKLOADS[3].names, WORKLOADS[3].dims))
    tp = dict(zip(WORKLOADS[6].names, WORKLOADS[6].dims))
    for name in ("wq", "wk", "wv", "w1", "w3"):
        assert (8 * tp[name][0], tp[name][1]) == full[name], name
    for name in ("wo", "w2"):
        assert (tp[name][0], 8 * tp[name][1]) == full[name], name
    for name in ("attention_norm", "ffn_norm"):
        assert tp[name] == full[name]
    assert WORKLOADS[6].world_size == 8


def test_uneven_workload():
    wl = WORKLOADS[5]
    assert wl.num_params == 40
    assert wl.dims[:3] == ((128256, 4096), (128256, 4096), (4096, 1))
    odd = wl.dims[3:]
    assert all(1 <= n <= 5000 and k in (1, 4096) for n, k in odd)
    assert sum(k == 1 for _, k in odd) == 18


def test_slabs_are_slices_of_the_full_tensor():
    full = param_rows(9, 2, 0, 300, 5000)
    assert full.dtype == np.float32 and full.shape == (300, 5000)
    for lo, hi in ((0, 1), (17, 211), (209, 300), (299, 300), (5, 5)):
        assert np.array_equal(param_rows(9, 2, lo, hi, 5000), full[lo:hi])
    g = grad_rows_bits(9, 3, 1, 0, 700, 3000)
    assert g.dtype == np.uint16
    assert np.array_equal(grad_rows_bits(9, 3, 1, 350, 701, 3000)[:350], g[350:])
    assert not np.array_equal(grad_rows_bits(9, 4, 1, 0, 10, 3000), g[:10])


def test_norms_are_one_and_values_are_scaled_normals():
    assert np.all(param_rows(3, 7, 0, 64, 1, is_norm=True) == 1.0)
    x = param_rows(3, 0, 0, 512, 512)
    assert abs(float(x.std()) - 0.02) < 0.001 and abs(float(x.mean())) < 0.001
    g = grad_rows_bits(3, 0, 0, 0, 512, 512)
    gf = (g.astype(np.uint32) << 16).view(np.float32)
    assert abs(float(gf.std()) - 1e-3) < 1e-4


def test_random_bits_deterministic():
    assert np.array_equal(random_bits16([1, 2], 1000), random_bits16([1, 2], 1000))
    assert not np.array_equal(random_bits16([1, 2], 1000), random_bits16([1, 3], 1000))


def test_workload_sizes_match_the_worked_table():
    """E, S and W*S of every workload, from the oracle's planner and the
    library's, against tests/golden/workload_sizes.txt."""
    import oracle.fsdp_oracle as O
    rows = [[int(x) for x in r] for r in read_table("workload_sizes.txt")]
    for key, W, P, E, S, WS in rows:
        wl = WORKLOADS[key]
        assert (wl.world_size, wl.num_params, wl.total_elems) == (W, P, E)
        plan = O.make_plan(W, wl.dims, 8)
        assert plan.chunk == S and W * S == WS
        if key != 5:
            assert WS == E
        try:
            from paper_2411_00284_amd import BucketPlan
        except ImportError:
            continue
        bp = BucketPlan(W, wl.dims, 8)
        assert bp.chunk_elems == S
        bp.close()
