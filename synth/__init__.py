"""Seeded synthetic workloads for the bucketed FSDP copy path.

This package only describes *inputs*: the parameter shapes of the five
workloads and seeded generators for parameter values, gradient values and raw
bit patterns.  It holds none of the method's arithmetic (no planning, packing,
casting with round-to-nearest-even, or reduction), so both the CPU oracle and
the GPU path can draw the same inputs from it without sharing any code that
computes a result.

Shapes follow the Llama 3.1 model table of the paper (Table 2: model and FFN
dimensions of the 8B, 70B and 405B models); the key/value projection height
(8 KV heads x 128 = 1024 rows) and the 128256-entry vocabulary are the
standard Llama-3 values.  Parameter order inside a transformer block is
wq, wk, wv, wo, w1, w2, w3, attention_norm, ffn_norm.
"""

from .workloads import WORKLOADS, Workload, workload
from .values import (
    param_rows,
    grad_rows_bits,
    random_bits16,
    random_bits32,
    exact_grad_bits,
)

__all__ = [
    "WORKLOADS",
    "Workload",
    "workload",
    "param_rows",
    "grad_rows_bits",
    "random_bits16",
    "random_bits32",
    "exact_grad_bits",
]
