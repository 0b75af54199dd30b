"""CPU oracle for the composed-prefill hot path.  TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously correct NumPy (fp64 where the math is
floating point) restatement of what the path computes, written from the
paper's definitions.  Only the tests, the smoke check and the benchmark's CPU
baseline leg may import it; the product library never does, and it shares no
code with the GPU path.

Modules and what each follows:

* layout     -- prompt placement before preparation and the compute / gather
                / retain sets (Section 5.3 "Placement before preparation",
                "Completing prefill"; Section 5.1 "Storage blocks").
* rope       -- rotary position encoding of keys and queries, and its
                re-application to keys cached before RoPE (Section 2.2).
* numerics   -- rounding to bf16 and OCP e4m3 storage formats.
* compose    -- assembling a request's KV from cached unit states, appending
                freshly computed tokens, retaining computed units (Sections
                5.3, 5.4).
* attention  -- causal GQA prefill attention over the assembled KV for the
                tokens that are computed (Section 5.3 "Completing prefill").
* pipeline   -- the whole per-layer path on a workload, and a dense full
                prefill used as a reference point.
* control    -- retrieval-aware scoring, admission, eviction and routing,
                and their trace replay (Section 5.2).

Every function is pinned by tests/test_oracle_*.py against closed forms,
library routines, brute force on tiny inputs, and the paper's worked
examples.  Parity status per function is listed in each module docstring.
"""
from . import attention, compose, control, layout, numerics, pipeline, rope  # noqa: F401
