"""The auto-wrapping oracle against its pins (no GPU), and each planted
mistake caught by at least one of them."""

from __future__ import annotations

import pytest

import auto_wrap_checks as C
from oracle.auto_wrap import auto_wrap, bucket_index, comm_time


def test_oracle_passes_every_pin():
    C.run_all(auto_wrap)


def test_bucket_index():
    assert bucket_index([[0], [1, 2], [3]]) == [0, 1, 1, 2]
    assert bucket_index([]) == []


def test_simulation_matches_hand_worked_timeline():
    """The timeline simulation on golden case B1 as cut by hand.  Step 0 waits
    for AG(B_0) = 1 + 2; steps 1 and 2 wait for nothing; step 3 waits
    RS(B_1) + AG(B_3) - T_c(B_2) = (1 + 2*5) + (1 + 3) - 2; step 4 waits
    RS(B_2) + AG(B_4) - T_c(B_3) = (1 + 2*3) + (1 + 1) - 1."""
    c = next(x for x in C.read_cases() if x["name"] == "B1")
    stalls, mems = C.simulate(c["expect"], c["ag"], c["rs"], c["t"], c["m"], c["alpha_ag"], c["beta_ag"],
                              c["alpha_rs"], c["beta_rs"], True)
    assert stalls == [3.0, 0.0, 0.0, 13.0, 8.0]
    assert stalls[0] == comm_time(1, 1, 2)
    assert mems == [0, 0, 0, 0, 0]


# ------------------------------------------------------------------- mutants

def _mutant(**flags):
    """A copy of the greedy walk with one planted mistake (selected by flag)."""
    def wrap(ag, t, m, alpha_ag, beta_ag, mem_max, backward=False, rs=None, alpha_rs=0.0, beta_rs=0.0):
        closed, cur, mem_acc = [], [], 0
        for i in range(len(ag)):
            if not cur:
                cur = [i]
                continue
            if flags.get("tc_of_current"):
                src = cur
            else:
                src = closed[-1] if closed else []
            if flags.get("tc_skips_last") and src:
                src = src[:-1]
            T_c = 0.0
            for j in src:
                T_c += t[j]
            if flags.get("first_free") and not closed:
                T_c = float("inf")
            words = sum(ag[j] for j in cur) + ag[i]
            if flags.get("alpha_per_node"):
                T_ag = sum(alpha_ag + beta_ag * ag[j] for j in cur) + alpha_ag + beta_ag * ag[i]
            else:
                T_ag = alpha_ag + beta_ag * words
            T_rs = 0.0
            if backward and not flags.get("drop_rs"):
                back = 1 if flags.get("rs_of_last") else 2
                rs_src = closed[-back] if len(closed) >= back else None
                if rs_src is not None:
                    T_rs = alpha_rs + beta_rs * sum(rs[j] for j in rs_src)
            M_c = sum(m[j] for j in cur)
            if flags.get("mem_no_reset"):
                M_c += mem_acc
            time_ok = (T_rs + T_ag < T_c) if flags.get("strict") else (T_rs + T_ag <= T_c)
            mem_ok = (M_c <= mem_max) if flags.get("mem_without_mi") else (M_c + m[i] <= mem_max)
            if time_ok and mem_ok:
                cur.append(i)
            else:
                mem_acc += sum(m[j] for j in cur)
                closed.append(cur)
                cur = [i]
        if cur:
            closed.append(cur)
        return closed
    return wrap


MUTANTS = {
    "strict time comparison": dict(strict=True),
    "backward ignores the reduce-scatter": dict(drop_rs=True),
    "reduce-scatter of the wrong bucket": dict(rs_of_last=True),
    "T_c of the bucket being built": dict(tc_of_current=True),
    "T_c misses a node": dict(tc_skips_last=True),
    "first bucket grows freely": dict(first_free=True),
    "alpha paid per node": dict(alpha_per_node=True),
    "memory check without M_ci": dict(mem_without_mi=True),
    "memory not reset per bucket": dict(mem_no_reset=True),
}


def test_unmutated_copy_passes():
    C.run_all(_mutant(), quick=True)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    with pytest.raises(AssertionError):
        C.run_all(_mutant(**MUTANTS[name]), quick=True)
