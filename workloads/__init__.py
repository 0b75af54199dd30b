"""Seeded synthetic inputs for the composed-prefill path.

This package only draws inputs: request structure (ordered context units,
their lengths, residency, recompute windows, page ids) and the values of the
cached unit states and fresh per-token projections.  It contains none of the
method's arithmetic (no RoPE, no gather, no attention), so that both the CPU
oracle and the GPU path can consume the same inputs without sharing code.
"""
from .configs import CONFIGS, ModelShape, WorkloadConfig, get_config
from .generate import (HIT, MISS, RequestSpec, UnitRef, Workload, generate,
                       make_workload)

__all__ = [
    "CONFIGS", "ModelShape", "WorkloadConfig", "get_config",
    "HIT", "MISS", "RequestSpec", "UnitRef", "Workload", "generate",
    "make_workload",
]
