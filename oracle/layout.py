"""Prompt layout and the token sets of composed prefill.

Follows Section 5.3 ("Placement before preparation": the prompt layout and
the request's KV slots are fixed before any unit is prepared; "Completing
prefill": the ranges selected by the composition policy are recomputed and
the remaining prompt -- separators, query -- is processed in one final
extend pass) and Section 5.1 ("Storage blocks": a unit of n tokens occupies
ceil(n/B) blocks that need not be adjacent).

Readings (the paper does not spell these out):
* segments are placed contiguously in prompt order from position 0
  (instruction, then units in retrieval order, then the query);
* the composition policy is EPIC's fixed chunk-initial window (Section 7):
  the first min(r, n) tokens of every reused unit are recomputed;
* with GLOBAL miss scope, every token of a computed (MISS) unit is a row of
  the final causal pass over the whole assembled prompt;
* with LOCAL miss scope (the paper's own semantics, Section 5.3: missing
  units are prefilled independently, then composed like hits), a MISS
  unit's tokens past its recompute window see only the keys of their own
  unit; the window (the first min(r, n) tokens, as for a HIT) and the text
  tokens are rows of the final pass over the whole prompt.  The unit's
  independent prefill is evaluated at its final positions: by the relative
  property of RoPE this equals a prefill from position 0 (pinned).

Pins: the worked example of Section 2.2 (Doc B at positions 150-249 in one
prompt and 50-149 in the other), ceil(n/B) page counts, and set algebra
(compute and gather sets partition the prompt).
"""
from __future__ import annotations

import numpy as np

MISS = 0
HIT = 1


def pages_for(n_tokens: int, page_size: int) -> int:
    """Number of fixed-size storage blocks a unit of n tokens occupies."""
    return -(-int(n_tokens) // int(page_size))


def layout(lengths) -> list[int]:
    """Start positions of segments placed contiguously in order from 0."""
    starts, p = [], 0
    for n in lengths:
        starts.append(p)
        p += int(n)
    return starts


def segments(req) -> list[tuple[str, int, int, object]]:
    """The request's segments in prompt order: (kind, start, length, unit)."""
    segs = [("text", int(s), int(n), None) for s, n in req.text_segs if n > 0]
    segs += [("unit", int(u.position), int(u.n_tokens), u) for u in req.units]
    segs.sort(key=lambda t: t[1])
    return segs


def check_tiling(req) -> None:
    """Raise ValueError unless the segments tile [0, prompt_len) once, in order."""
    p = 0
    for kind, s, n, _ in segments(req):
        if s != p or n <= 0:
            raise ValueError(f"segment at {s} (len {n}) breaks tiling at {p}")
        p += n
    if p != req.prompt_len:
        raise ValueError(f"segments cover {p} tokens, prompt_len={req.prompt_len}")


def recompute_count(u) -> int:
    """Leading tokens of a unit computed in the final pass."""
    if u.residency == MISS:
        return int(u.n_tokens)
    return min(int(u.n_recompute), int(u.n_tokens))


def compute_positions(req) -> np.ndarray:
    """Sorted prompt positions of the tokens computed in the final pass."""
    pos = []
    for kind, s, n, u in segments(req):
        if kind == "text":
            pos.extend(range(s, s + n))
        else:
            pos.extend(range(s, s + recompute_count(u)))
    return np.asarray(sorted(pos), dtype=np.int64)


GLOBAL = 0
LOCAL = 1


def miss_scope(req) -> int:
    """GLOBAL (default) or LOCAL miss scope of a request."""
    return int(getattr(req, "miss_scope", GLOBAL))


def row_kv_lo(req) -> np.ndarray:
    """First visible key position of every computed row (compute_positions
    order): 0, except under LOCAL scope for a MISS unit's tokens past its
    recompute window, which see only their own unit."""
    pos = compute_positions(req)
    lo = np.zeros(len(pos), dtype=np.int64)
    if miss_scope(req) != LOCAL:
        return lo
    for u in req.units:
        if u.residency != MISS:
            continue
        r = min(int(u.n_recompute), int(u.n_tokens))
        start, end = int(u.position) + r, int(u.position) + int(u.n_tokens)
        sel = (pos >= start) & (pos < end)
        lo[sel] = int(u.position)
    return lo


def gather_tokens(req) -> list[tuple[int, int, int]]:
    """(unit index, token j, prompt position) of every cached token reused."""
    out = []
    for ui, u in enumerate(req.units):
        if u.residency != HIT:
            continue
        for j in range(recompute_count(u), int(u.n_tokens)):
            out.append((ui, j, int(u.position) + j))
    return out


def retain_tokens(req, page_size: int) -> list[tuple[int, int, int, int, int]]:
    """(unit index, j, position, pool page, slot) written back to the pool.

    Token j of a unit lives in block j // B at slot j % B (Section 5.1).
    """
    out = []
    for ui, u in enumerate(req.units):
        if u.residency != MISS or not u.retain:
            continue
        for j in range(int(u.n_tokens)):
            out.append((ui, j, int(u.position) + j,
                        int(u.pool_pages[j // page_size]), j % page_size))
    return out


def slot_of(block_table, position: int, page_size: int) -> tuple[int, int]:
    """(request page, slot) of a prompt position through the block table."""
    return int(block_table[position // page_size]), position % page_size


def kv_bytes_per_token(n_layers: int, n_kv_heads: int, head_dim: int,
                       elem_bytes: int, tp: int = 1) -> int:
    """Bytes of KV state one token produces per rank (Section 2.4):
    keys and values (2) for every layer, for the rank's H_kv / TP heads."""
    if n_kv_heads % tp:
        raise ValueError("H_kv must divide evenly across TP ranks")
    return 2 * n_layers * (n_kv_heads // tp) * head_dim * elem_bytes
