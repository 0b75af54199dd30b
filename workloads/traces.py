"""Seeded synthetic retrieval traces for the control plane.

A trace is a sequence of requests, each the ordered list of context units a
retriever returned, with every unit's token count.  Unit popularity is Zipf
over a fixed universe, optionally drifting (the popular set shifts every
`drift_every` requests), the shape of the paper's retrieval workloads
(Section 3: recurrence beyond the prompt prefix).  Values only: nothing here
scores, admits, evicts or routes.
"""
from __future__ import annotations

import numpy as np

_TAG_TRACE = 0x7EACE


def zipf_trace(seed: int, n_requests: int, n_units: int, units_per_request: int,
               zipf_s: float = 1.0, token_range=(64, 512), drift_every: int = 0,
               drift_shift: int = 0):
    """Returns a list of (unit_ids, unit_tokens) pairs (numpy arrays)."""
    rng = np.random.default_rng((seed, _TAG_TRACE))
    lengths = rng.integers(token_range[0], token_range[1] + 1, size=n_units).astype(np.int32)
    w = np.arange(1, n_units + 1, dtype=np.float64) ** (-zipf_s)
    p = w / w.sum()
    out = []
    for i in range(n_requests):
        k = min(units_per_request, n_units)
        ranks = rng.choice(n_units, size=k, replace=False, p=p)
        shift = (i // drift_every) * drift_shift if drift_every else 0
        ids = ((ranks + shift) % n_units).astype(np.uint64)
        out.append((ids, lengths[ids.astype(np.int64)]))
    return out
