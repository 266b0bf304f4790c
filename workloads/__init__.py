"""Seeded synthetic inputs for the batched speculative-verification step.

This package only draws random numbers and lays them out in memory.  It is
shared by the CPU oracle's tests and by the GPU path's tests and benchmark so
that both consume bit-identical inputs; it computes none of the verification
arithmetic (no attention, no log-sum-exp, no acceptance test, no resampling).

The draft distributions ``q`` are produced by a stand-in for the draft model
M_q (it sits outside the verification step): for the correlated recipes it
perturbs a plain float32 product of the synthetic hidden states and vocabulary
weights, see :func:`workloads.generate.draft_logits_f32`.
"""

from .configs import CONFIGS, Workload, get_config
from .generate import (
    VerifyInputs,
    bf16_bits,
    bf16_round,
    make_inputs,
)

__all__ = [
    "CONFIGS",
    "Workload",
    "get_config",
    "VerifyInputs",
    "bf16_bits",
    "bf16_round",
    "make_inputs",
]
