"""CPU oracle for SimpleFSDP's auto-wrapping decision.

TEST INFRASTRUCTURE ONLY.  This module is the plain definition that the
library's host planner (``fsdp_auto_wrap``) is checked against.  Only the test
suite may import it; it shares no code with the library.

What is computed (SimpleFSDP, arXiv 2411.00284, section 3.3.2
"Auto-wrapping": the profiling model, Algorithm 1 and the variables of
Table 1):

* A pass issues one all-gather (AG) per parameter node i = 0..n-1, in the
  order the pass computes the nodes (the forward pass in model order, the
  backward pass in its own, usually reversed, order).  Auto-wrapping cuts
  this sequence into consecutive buckets B_0, B_1, ...; step k computes the
  nodes of B_k.
* With the reordering of section 3.2.2, the all-gather of B_{k+1} is in
  flight while step k computes; in the backward pass so is the
  reduce-scatter (RS) of the gradients step k-1 produced, the bucket B_{k-1}.
* A collective that moves n words costs T_m = alpha + beta * n (the
  profiling model); a bucketed collective moves the sum of its nodes' words,
  so bucketing pays alpha once per bucket.
* Node i joins the bucket B being built (the bucket after the last closed
  one, B_k) exactly when Algorithm 1 says so:
    forward   T^AG_(m+mi) <= T_c                  and  M_c + M_ci <= M_max
    backward  T^RS_m + T^AG_(m+mi) <= T_c         and  M_c + M_ci <= M_max
  with (Table 1) T^AG_(m+mi) = alpha_AG + beta_AG * (words of B + n_i),
  T_c = the compute time of step k (the sum of T_cj over B_k),
  M_c = the peak compute memory of B so far (the sum of M_cj over B),
  T^RS_m = alpha_RS + beta_RS * (RS words of B_{k-1}).
  Otherwise B is closed and node i starts the next bucket alone.

Readings where the paper is silent:

* The first bucket's all-gather overlaps no computation: for B_0, T_c = 0.
  With alpha_AG > 0 it therefore holds one node.
* When there is no B_{k-1} (building B_1), no reduce-scatter is in flight:
  T^RS_m = 0.
* A node that starts a bucket is placed there whatever its own cost: the
  algorithm decides only whether a node joins the previous one.
* M_c adds the peak memories of the bucket's nodes (the paper writes
  M_c + M_c(i)).
* Arithmetic: words and memory are integers summed exactly; T_c is the sum,
  in node order from 0.0, of binary64 times; T_m = alpha + beta * float(n)
  with the product and the sum each rounded (no fused multiply-add); the
  backward left-hand side is T^RS_m + T^AG_(m+mi).  Every comparison is
  binary64 ``<=``.
"""

from __future__ import annotations

from typing import Sequence

__all__ = ["comm_time", "bucket_decision", "auto_wrap", "bucket_index"]


def comm_time(alpha: float, beta: float, words: int) -> float:
    """The profiling model of a collective moving ``words`` words:
    T_m = alpha + beta * n (section 3.3.2, "Profiling")."""
    return float(alpha) + float(beta) * float(words)


def bucket_decision(is_forward: bool, T_m_AG_merged: float, T_c: float, M_c: int, M_ci: int,
                    M_max: int, T_m_RS: float = 0.0) -> bool:
    """Algorithm 1: True to bucket the i-th all-gather with the previous
    ones, False to start a new bucket (variables of Table 1)."""
    if is_forward:
        time_constraint = T_m_AG_merged <= T_c
    else:
        time_constraint = T_m_RS + T_m_AG_merged <= T_c
    mem_constraint = M_c + M_ci <= M_max
    return time_constraint and mem_constraint


def auto_wrap(ag_words: Sequence[int], compute_time: Sequence[float], compute_mem: Sequence[int],
              alpha_ag: float, beta_ag: float, mem_max: int, backward: bool = False,
              rs_words: Sequence[int] | None = None, alpha_rs: float = 0.0,
              beta_rs: float = 0.0) -> list[list[int]]:
    """Greedy auto-wrapping of one pass: the buckets, as lists of node
    indices, in order.

    ``ag_words[i]``, ``compute_time[i]`` and ``compute_mem[i]`` are n_i,
    T_ci and M_ci of node i; ``rs_words[i]`` (backward only) is the words of
    its gradient's reduce-scatter.
    """
    n = len(ag_words)
    assert len(compute_time) == n and len(compute_mem) == n
    if backward:
        assert rs_words is not None and len(rs_words) == n
    closed: list[list[int]] = []      # B_0 .. B_k
    current: list[int] = []           # the bucket being built, B_{k+1}
    for i in range(n):
        if not current:
            current = [i]
            continue
        # T_c: step k's computation, i.e. the last closed bucket (none for B_0).
        T_c = 0.0
        if closed:
            for j in closed[-1]:
                T_c += float(compute_time[j])
        words = sum(int(ag_words[j]) for j in current) + int(ag_words[i])
        T_m_AG_merged = comm_time(alpha_ag, beta_ag, words)
        M_c = sum(int(compute_mem[j]) for j in current)
        T_m_RS = 0.0
        if backward and len(closed) >= 2:
            # the reduce-scatter of the bucket computed one step before step k
            T_m_RS = comm_time(alpha_rs, beta_rs, sum(int(rs_words[j]) for j in closed[-2]))
        if bucket_decision(not backward, T_m_AG_merged, T_c, M_c, int(compute_mem[i]), int(mem_max), T_m_RS):
            current.append(i)
        else:
            closed.append(current)
            current = [i]
    if current:
        closed.append(current)
    return closed


def bucket_index(buckets: Sequence[Sequence[int]]) -> list[int]:
    """The bucket number of every node, from a list of buckets."""
    out = [0] * sum(len(b) for b in buckets)
    for k, b in enumerate(buckets):
        for i in b:
            out[i] = k
    return out
