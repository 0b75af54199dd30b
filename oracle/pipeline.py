"""The whole per-layer composed-prefill path on a workload (oracle).

compose (gather + re-rotation of cached hits) -> append (fresh tokens rotated
at their positions) -> causal GQA attention for the computed tokens ->
retention of computed units in their reusable form.  Section 5.3 and 5.4.

`full_prefill` is the dense causal prefill of the same prompt in which every
token is computed; with every token recomputed the composed path must equal
it (pinned in tests/test_oracle_pipeline.py).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import layout as L
from .attention import causal_gqa_attention
from .compose import (assemble_request_kv, assemble_request_kv_e4m3, dequantize,
                      quantized_queries_e4m3, retained_pages, round_storage,
                      rotated_queries)
from .rope import rope_fp32


@dataclass
class RequestResult:
    positions: np.ndarray      # compute-token positions, plan order
    K: np.ndarray              # assembled rotated keys [P][h_kv][d] (float32 values)
    V: np.ndarray              # assembled values [P][h_kv][d]
    source: np.ndarray         # per position: 'gather' | 'compute'
    q: np.ndarray              # rotated queries [T_r][h_q][d] (float32 values)
    out: np.ndarray            # fp64 [T_r][h_q][d]
    lse: np.ndarray            # fp64 [T_r][h_q]
    kv_heads: np.ndarray
    q_heads: np.ndarray
    kv_lo: np.ndarray          # first visible key of every row


def run_request(wl, r: int, kv_heads=None, scale=None) -> RequestResult:
    m = wl.model
    G = m.n_q_heads // m.n_kv_heads
    kvh = np.arange(m.n_kv_heads) if kv_heads is None else np.asarray(kv_heads)
    qh = np.concatenate([np.arange(g * G, (g + 1) * G) for g in kvh])
    if m.kv_dtype == "e4m3":
        Kc, Vc, ks, vs = assemble_request_kv_e4m3(wl, r)
        K = (dequantize(Kc, 1.0) * ks[:, None, None])[:, kvh]
        V = (dequantize(Vc, 1.0) * vs[:, None, None])[:, kvh]
        src = None
        cpos, q = quantized_queries_e4m3(wl, r, qh)
    else:
        K, V, src = assemble_request_kv(wl, r, kvh)
        cpos, q = rotated_queries(wl, r, qh)
    lo = L.row_kv_lo(wl.requests[r])
    out, lse = causal_gqa_attention(q, cpos, K, V, scale=scale, kv_lo=lo)
    return RequestResult(cpos, K, V, src, q, out, lse, kvh, qh, lo)


def run(wl, requests=None, kv_heads=None, scale=None):
    """Oracle results per request (list), and the retained pool pages."""
    from .compose import retained_pages_e4m3
    reqs = range(len(wl.requests)) if requests is None else requests
    results = {r: run_request(wl, r, kv_heads, scale) for r in reqs}
    kept = retained_pages_e4m3(wl) if wl.model.kv_dtype == "e4m3" else retained_pages(wl)
    return results, kept


def full_prefill(wl, r: int, scale=None):
    """Dense causal prefill of request r with every token computed.

    Uses the fresh projections at every prompt position; keys and queries
    rotated at their positions exactly as computed tokens are.
    """
    m = wl.model
    P = wl.requests[r].prompt_len
    pos = np.arange(P)
    q, k, v = wl.fresh(r, pos)
    qr = round_storage(rope_fp32(q, pos, m.rope_theta), m.act_dtype)
    kr = round_storage(rope_fp32(k, pos, m.rope_theta), m.kv_dtype)
    return causal_gqa_attention(qr, pos, kr, v, scale=scale)


def unit_prefill(wl, r: int, ui: int, scale=None):
    """Independent causal prefill of unit ui of request r from position 0
    (its tokens only, rotated at 0 .. n-1), as the paper prepares a missing
    unit (Section 5.3); used to pin the LOCAL miss scope."""
    m = wl.model
    u = wl.requests[r].units[ui]
    n = int(u.n_tokens)
    q, k, v = wl.fresh(r, np.arange(u.position, u.position + n))
    pos = np.arange(n)
    qr = round_storage(rope_fp32(q, pos, m.rope_theta), m.act_dtype)
    kr = round_storage(rope_fp32(k, pos, m.rope_theta), m.kv_dtype)
    return causal_gqa_attention(qr, pos, kr, v, scale=scale)


def counts(wl):
    """Algorithmic counts of the path on a workload (per layer).

    gather_tokens, compute_tokens, retain_tokens, prompt_tokens, and the
    attention's visible (row, key) pairs summed over compute rows.
    """
    g = c = rt = vis = 0
    for req in wl.requests:
        g += len(L.gather_tokens(req))
        cp = L.compute_positions(req)
        c += len(cp)
        vis += int((cp - L.row_kv_lo(req) + 1).sum())
        rt += len(L.retain_tokens(req, wl.model.page_size))
    return dict(gather_tokens=g, compute_tokens=c, retain_tokens=rt,
                prompt_tokens=wl.prompt_tokens, visible_pairs=vis)
