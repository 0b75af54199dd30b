"""Assembling a request's KV from cached unit states (oracle).

Follows Section 5.3: cache hits are placed into the request's KV slots with
RoPE applied to the keys at their new positions; missing units and the
remaining prompt are computed (their keys rotated at their own positions);
the composition policy's recompute window replaces the first tokens of each
reused unit with freshly computed states, used only by this request.
Section 5.4 / 5.1: what is retained is the reusable form -- keys before RoPE
and values -- written into the unit's storage blocks, token j in block j // B
at slot j % B.

Precision semantics (documented readings, mirrored by the GPU path):
* keys are rotated with rope_fp32 (fp32 table, no FMA) and rounded once to
  the KV storage dtype; values are copied bit for bit;
* fresh queries are rotated the same way and rounded to the activation dtype,
  which is what the attention contraction consumes.

The assembled KV is returned in logical form, one row per prompt position
([P][H_kv][d]); paging is addressing only and is checked by the tests through
the block table.  Parity: pinned (gather bit-exact by definition; rotation
pinned through oracle.rope; set algebra through oracle.layout).
"""
from __future__ import annotations

import numpy as np

from . import layout as L
from .numerics import round_bf16
from .rope import rope_fp32


def round_storage(x, dtype: str) -> np.ndarray:
    """Round fp32 values to a storage dtype, returned as float32."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32)
    if dtype == "bf16":
        return round_bf16(x)
    raise ValueError(f"unsupported storage dtype {dtype!r}")


def assemble_request_kv(wl, r: int, kv_heads=None):
    """Assembled K (rotated) and V of request r, [prompt_len][h][d] each.

    Returns (K, V, source) where source[p] is 'gather' or 'compute'.
    `kv_heads` restricts the output to a subset of KV heads (for sampling).
    """
    m = wl.model
    req = wl.requests[r]
    L.check_tiling(req)
    heads = np.arange(m.n_kv_heads) if kv_heads is None else np.asarray(kv_heads)
    P = req.prompt_len
    K = np.full((P, len(heads), m.head_dim), np.nan, dtype=np.float32)
    V = np.full((P, len(heads), m.head_dim), np.nan, dtype=np.float32)
    source = np.empty(P, dtype=object)

    # cached hits: gather + re-rotate to the unit's new positions
    for ui, u in enumerate(req.units):
        if u.residency != L.HIT:
            continue
        j0 = L.recompute_count(u)
        if j0 >= u.n_tokens:
            continue
        k_pre, v = wl.unit_state(u.unit_id)
        j = np.arange(j0, u.n_tokens)
        pos = u.position + j
        K[pos] = round_storage(rope_fp32(k_pre[j][:, heads], pos, m.rope_theta),
                               m.kv_dtype)
        V[pos] = v[j][:, heads]
        source[pos] = "gather"

    # computed tokens: fresh k rotated at its own position, v as is
    cpos = L.compute_positions(req)
    if cpos.size:
        _, k, v = wl.fresh(r, cpos)
        K[cpos] = round_storage(rope_fp32(k[:, heads], cpos, m.rope_theta),
                                m.kv_dtype)
        V[cpos] = v[:, heads]
        source[cpos] = "compute"
    return K, V, source


def rotated_queries(wl, r: int, q_heads=None):
    """Fresh queries of request r's compute tokens, rotated and rounded."""
    m = wl.model
    cpos = L.compute_positions(wl.requests[r])
    q, _, _ = wl.fresh(r, cpos)
    if q_heads is not None:
        q = q[:, np.asarray(q_heads)]
    return cpos, round_storage(rope_fp32(q, cpos, m.rope_theta), m.act_dtype)


def retained_pages(wl):
    """Pool blocks written by retention, as {page: (k, v, filled)}.

    k, v are [H_kv][B][d] float32 (the pre-RoPE fresh values, bit copies);
    filled[s] tells which slots of the page the unit covers -- the others
    are left untouched.
    """
    m = wl.model
    B = m.page_size
    out = {}
    for r, req in enumerate(wl.requests):
        toks = L.retain_tokens(req, B)
        if not toks:
            continue
        pos = np.array([t[2] for t in toks])
        _, k, v = wl.fresh(r, pos)
        for (ui, j, p, page, slot), kr, vr in zip(toks, k, v):
            if page not in out:
                out[page] = (np.zeros((m.n_kv_heads, B, m.head_dim), np.float32),
                             np.zeros((m.n_kv_heads, B, m.head_dim), np.float32),
                             np.zeros(B, dtype=bool))
            pk, pv, filled = out[page]
            if filled[slot]:
                raise ValueError(f"pool page {page} slot {slot} retained twice")
            pk[:, slot] = kr
            pv[:, slot] = vr
            filled[slot] = True
    return out
