"""Seeded synthetic inputs for CURE's verify-and-repair step.

This module serves both sides of every parity check (the HIP path and the CPU
oracle) and holds none of the method's arithmetic: it draws random numbers,
quantises them to the storage type and plants structure (tree shape, target
argmax, logit gaps, ranked heads of draft rows) by construction. No margin,
ranking, softmax or acceptance is computed here.
"""

from .workloads import (
    Workload, make_workload, preset, PRESETS, bf16_round, bf16_ceil,
    algorithmic_bytes,
)
from .draft import DraftBlock, make_draft_block

__all__ = ["Workload", "make_workload", "preset", "PRESETS", "bf16_round",
           "bf16_ceil", "algorithmic_bytes", "DraftBlock", "make_draft_block"]
