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


# ------------------------------------------------------------------ e4m3 pool
# Readings (the paper has no 8-bit path): the pool holds e4m3 codes with one
# power-of-two fp32 scale per (page, K|V); a value is decode(code) * scale.
# Request pages use the same format.  Every request page has one writer:
#   gathered page   V codes and scale copied; K dequantized, rotated to the
#                   new positions in fp32 (rope_fp32), and requantized with a
#                   fresh page scale (rotation can grow |x| by up to sqrt(2));
#   computed page   fresh k rotated in fp32 and v, each quantized per page;
# retention quantizes the unit's pre-RoPE k and v per pool page.  The page
# scale is the smallest power of two s with amax / s <= 448 over the page's
# valid tokens (all heads and dims); codes are nearest-even, saturating.

def quantize_page(x):
    """x [n][H][d] fp32 -> (codes uint8, scale fp32) with one page scale."""
    from .numerics import e4m3_encode, e4m3_page_scale
    x = np.asarray(x, dtype=np.float32)
    amax = float(np.abs(x).max()) if x.size else 0.0
    scale = np.float32(e4m3_page_scale(np.array([amax]))[0])
    return e4m3_encode(x / scale), scale


def dequantize(codes, scale):
    from .numerics import e4m3_decode
    return e4m3_decode(codes) * np.float32(scale)


def check_page_aligned(req, page_size: int) -> None:
    """Raise ValueError unless every request page has a single writer."""
    B = page_size
    for kind, s, n, u in L.segments(req):
        end = s + n
        if s % B or (end % B and end != req.prompt_len):
            raise ValueError(f"segment [{s}, {end}) is not page aligned")
        if u is not None and u.residency == L.HIT:
            r = L.recompute_count(u)
            if r % B and r != n:
                raise ValueError("recompute window is not page aligned")


def assemble_request_kv_e4m3(wl, r: int):
    """Request r's pages: per position K codes, V codes ([P][H][d] uint8) and
    the page scale of each position's page (k_scale[P], v_scale[P])."""
    m = wl.model
    B = m.page_size
    req = wl.requests[r]
    L.check_tiling(req)
    check_page_aligned(req, B)
    P = req.prompt_len
    Kc = np.zeros((P, m.n_kv_heads, m.head_dim), dtype=np.uint8)
    Vc = np.zeros_like(Kc)
    ks = np.zeros(P, dtype=np.float32)
    vs = np.zeros(P, dtype=np.float32)
    cpos = L.compute_positions(req)
    _, kf, vf = wl.fresh(r, cpos) if cpos.size else (None, None, None)
    row_of = {int(p): i for i, p in enumerate(cpos)}
    cache = {}
    for pg in range(-(-P // B)):
        p0, p1 = pg * B, min(P, (pg + 1) * B)
        pos = np.arange(p0, p1)
        if p0 in row_of:           # computed page
            rows = np.array([row_of[int(p)] for p in pos])
            kc, ksc = quantize_page(rope_fp32(kf[rows], pos, m.rope_theta))
            vc, vsc = quantize_page(vf[rows])
        else:                      # gathered page of a HIT unit
            u = next(u for u in req.units if u.position <= p0 < u.position + u.n_tokens)
            if u.unit_id not in cache:
                cache[u.unit_id] = wl.unit_state_e4m3(u.unit_id)
            kcodes, vcodes, kscale, vscale = cache[u.unit_id]
            j0 = p0 - u.position
            src = j0 // B
            j = np.arange(j0, j0 + (p1 - p0))
            kx = dequantize(kcodes[j], kscale[src])
            kc, ksc = quantize_page(rope_fp32(kx, pos, m.rope_theta))
            vc, vsc = vcodes[j], vscale[src]
        Kc[p0:p1], Vc[p0:p1], ks[p0:p1], vs[p0:p1] = kc, vc, ksc, vsc
    return Kc, Vc, ks, vs


def quantized_queries_e4m3(wl, r: int, q_heads=None):
    """Rotated fresh queries quantized per (row, head) with a power-of-two
    scale, as the fp8 attention consumes them (a kernel choice mirrored
    here).  Returns (positions, dequantized q [T][h][d] fp32)."""
    from .numerics import e4m3_decode, e4m3_encode, e4m3_page_scale
    m = wl.model
    cpos = L.compute_positions(wl.requests[r])
    q, _, _ = wl.fresh(r, cpos)
    if q_heads is not None:
        q = q[:, np.asarray(q_heads)]
    qr = rope_fp32(q, cpos, m.rope_theta)
    amax = np.abs(qr).max(axis=-1)                     # [T][h]
    sc = e4m3_page_scale(amax.ravel()).reshape(amax.shape)
    codes = e4m3_encode(qr / sc[..., None])
    return cpos, e4m3_decode(codes) * sc[..., None]


def retained_pages_e4m3(wl):
    """Pool blocks written by retention in the e4m3 pool:
    {page: (k_codes [H][B][d], v_codes, k_scale, v_scale, filled[B])}."""
    m = wl.model
    B = m.page_size
    out = {}
    for r, req in enumerate(wl.requests):
        for u in req.units:
            if u.residency != L.MISS or not u.retain:
                continue
            pos = np.arange(u.position, u.position + u.n_tokens)
            _, k, v = wl.fresh(r, pos)
            for pi, page in enumerate(u.pool_pages):
                j = np.arange(pi * B, min(u.n_tokens, (pi + 1) * B))
                kc, ksc = quantize_page(k[j])
                vc, vsc = quantize_page(v[j])
                kp = np.zeros((m.n_kv_heads, B, m.head_dim), np.uint8)
                vp = np.zeros_like(kp)
                filled = np.zeros(B, dtype=bool)
                kp[:, :len(j)] = kc.transpose(1, 0, 2)
                vp[:, :len(j)] = vc.transpose(1, 0, 2)
                filled[:len(j)] = True
                out[int(page)] = (kp, vp, ksc, vsc, filled)
    return out
