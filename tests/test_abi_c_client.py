"""The library's host entry points called from a plain C program (no Python
in between, no GPU): planner results and auto-wrapping cuts equal the
oracle's."""

from __future__ import annotations

import os
import subprocess

import pytest

import auto_wrap_checks as AW
import oracle.fsdp_oracle as O
from oracle.auto_wrap import auto_wrap, bucket_index
from synth import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2411_00284_amd")
LIB = os.path.join(PKG, "libfsdp_bucket.so")


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    if not os.path.exists(LIB):
        pytest.fail("library not built")
    exe = str(tmp_path_factory.mktemp("abi") / "abi_client")
    cmd = ["gcc", "-std=c99", "-O1", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
           f"-I{os.path.join(ROOT, 'include')}", "-I/opt/rocm/include",
           os.path.join(ROOT, "tests", "abi_client.c"), "-o", exe,
           f"-L{PKG}", "-lfsdp_bucket", f"-Wl,-rpath,{PKG}", "-L/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return exe


def _run(exe, text):
    res = subprocess.run([exe], input=text, capture_output=True, text=True, timeout=60)
    assert res.returncode == 0, res.stderr
    return res.stdout.splitlines()


def test_planner_from_c(client):
    cases = [(wl.world_size, list(wl.dims), 8) for wl in WORKLOADS.values()]
    cases += [(3, [(7, 3), (2, 5), (10, 1), (0, 4)], 1), (64, [(65, 1), (128, 2)], 16)]
    text = "".join(f"{w} {len(d)} {a} " + " ".join(f"{n} {k}" for n, k in d) + "\n" for w, d, a in cases)
    lines = iter(_run(client, text))
    for w, dims, a in cases:
        want = O.make_plan(w, dims, a)
        assert next(lines) == f"plan 0 S={want.chunk}"
        for p in range(len(dims)):
            rows = ",".join(str(O.local_rows(want, p, r)) for r in range(w))
            assert next(lines) == (f"param {p} c={want.rows_per_rank[p]} off={want.offset[p]} "
                                   f"L={want.seg[p]} rows={rows}")


def test_planner_errors_from_c(client):
    out = _run(client, "0 1 8 4 4\n4 1 3 4 4\n4 1 8 -1 4\n")
    assert out[0] == "plan 1 S=-1" and out[1].startswith("error ")
    assert out[2] == "plan 1 S=-1" and "power of two" in out[3]
    assert out[4] == "plan 1 S=-1" and "dim0" in out[5]


def test_auto_wrap_from_c(client):
    for c in AW.read_cases():
        n = len(c["ag"])
        text = (f"wrap {n} {int(c['backward'])} {c['alpha_ag']!r} {c['beta_ag']!r} {c['alpha_rs']!r} "
                f"{c['beta_rs']!r} {c['mem_max']}\n")
        text += "".join(f"{c['ag'][i]} {c['rs'][i]} {c['t'][i]!r} {c['m'][i]}\n" for i in range(n))
        out = _run(client, text)
        want = auto_wrap(c["ag"], c["t"], c["m"], c["alpha_ag"], c["beta_ag"], c["mem_max"], c["backward"],
                         c["rs"], c["alpha_rs"], c["beta_rs"])
        assert want == c["expect"]
        assert out == [f"wrap 0 buckets={len(want)} of=" + ",".join(str(b) for b in bucket_index(want))], c["name"]
    out = _run(client, "wrap 2 0 -1 0 0 0 5\n1 1 1 1\n1 1 1 1\n")
    assert out == ["wrap 1 buckets=-1 of="]
