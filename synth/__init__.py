"""Seeded synthetic streams for the acoustic-to-text KV step.

This package only draws inputs: stream structure (rows per unit, their
segment classes, positions and unit ids, per-stream budgets) and the Q/K/V
values of each step.  It holds none of the method's arithmetic (no rotary
embedding, no attention, no eviction) so that both the CPU oracle and the
GPU path can consume identical inputs without sharing any method code.
"""
from .streams import (  # noqa: F401
    SEG_PREFIX, SEG_ACOUSTIC, SEG_DELIM, SEG_TEXT, SEG_RESPONSE, SEG_NAMES,
    CONFIGS, WorkloadConfig, StreamSpec, UnitSpec, Workload, make_workload,
    step_values, bf16_round, bf16_bits, tiny_stream,
)
