"""Pins for the e4m3 retention and query quantization of the oracle (the
paper has no 8-bit path; these follow the documented readings: the reusable
form of Section 5.4 -- keys before RoPE, values -- quantized per pool page
with the smallest power-of-two scale, and rotated queries quantized per
(row, head) with the same scale rule).

The checks do not call the oracle's quantizer: the e4m3 value set is built
here from the OCP e4m3fn definition (4 exponent bits, bias 7, 3 mantissa
bits, subnormals, no infinities, S.1111.111 is NaN) and every code is
checked to be a nearest grid point of the exact value, and every scale
minimal, by brute force.  Planted mistakes at the end must each fail one of
them.
"""
import dataclasses

import numpy as np
import pytest

import workloads
from oracle import compose as C
from oracle import layout as L
from oracle.numerics import e4m3_decode
from oracle.rope import rope_fp32


def _e4m3_magnitudes() -> np.ndarray:
    """Every finite non-negative e4m3fn magnitude, from the format's fields."""
    vals = [m / 8.0 * 2.0 ** -6 for m in range(8)]             # exponent field 0
    for e in range(1, 16):
        for m in range(8):
            if e == 15 and m == 7:
                continue                                         # NaN pattern
            vals.append((1.0 + m / 8.0) * 2.0 ** (e - 7))
    return np.unique(np.array(vals))


_MAG = _e4m3_magnitudes()
_GRID = np.unique(np.concatenate([-_MAG, _MAG]))                 # 253 values


def _check_scale_minimal(amax: float, s: float) -> None:
    s = float(s)
    assert s > 0 and np.log2(s) == np.round(np.log2(s)), f"scale {s} not a power of two"
    if amax == 0:
        assert s == 1.0
        return
    assert amax / s <= 448.0, f"amax {amax} exceeds 448 * scale {s}"
    assert amax / (s / 2) > 448.0, f"scale {s} not minimal for amax {amax}"


def _check_nearest(y, x, s) -> None:
    """y (decoded, times s) is a nearest point of s * grid to x, elementwise;
    x is in range (|x| <= 448 s), so no saturation is involved."""
    x = np.asarray(x, np.float64)
    s = np.broadcast_to(np.asarray(s, np.float64), x.shape).ravel()
    x = x.ravel()
    y = np.asarray(y, np.float64).ravel()
    q = y / s
    # on the grid
    idx = np.searchsorted(_GRID, q)
    idx = np.clip(idx, 0, len(_GRID) - 1)
    assert np.all(_GRID[idx] == q), "a decoded value is not on the e4m3 grid"
    # nearest: no grid point is strictly closer to x / s
    t = x / s
    j = np.clip(np.searchsorted(_GRID, t), 1, len(_GRID) - 1)
    best = np.minimum(np.abs(_GRID[j] - t), np.abs(_GRID[j - 1] - t))
    bad = np.abs(q - t) > best
    assert not bad.any(), (f"{int(bad.sum())} codes are not nearest; first: x/s={t[bad][0]}, "
                           f"got {q[bad][0]}, nearest distance {best[bad][0]}")


def _retain_workload():
    # ragged unit lengths (last pages partly filled), several MISS units
    cfg = workloads.get_config("small_fp8").with_(
        unit_tokens=(20, 70), extra={}, hit_prob=0.4, seed=21)
    wl = workloads.make_workload(cfg)
    assert any(u.residency == L.MISS and u.retain and u.n_tokens % wl.model.page_size
               for req in wl.requests for u in req.units)
    # fresh states whose magnitude changes by powers of two from one 16-token
    # block of positions to the next, so that neighbouring pages of a unit
    # need different scales (the bf16 values stay exactly representable)
    base = wl.fresh
    B = wl.model.page_size

    def fresh(req, positions):
        q, k, v = base(req, positions)
        f = np.ldexp(np.float32(1.0), (np.asarray(positions) // B) % 4 - 1)[:, None, None]
        return q * f, k * f, v * f
    return dataclasses.replace(wl, fresh_fn=fresh)


def _retained_units(wl):
    """(request, unit) of every retained MISS unit, in the oracle's order."""
    return [(r, u) for r, req in enumerate(wl.requests) for u in req.units
            if u.residency == L.MISS and u.retain]


def check_retained_scales_minimal(wl):
    pages = C.retained_pages_e4m3(wl)
    B = wl.model.page_size
    for r, u in _retained_units(wl):
        _, k, v = wl.fresh(r, np.arange(u.position, u.position + u.n_tokens))
        for pi, page in enumerate(u.pool_pages):
            j = slice(pi * B, min(u.n_tokens, (pi + 1) * B))
            _, _, ks, vs, _ = pages[int(page)]
            _check_scale_minimal(float(np.abs(k[j]).max()), ks)
            _check_scale_minimal(float(np.abs(v[j]).max()), vs)


def check_retained_codes_nearest_pre_rope(wl):
    pages = C.retained_pages_e4m3(wl)
    B = wl.model.page_size
    for r, u in _retained_units(wl):
        _, k, v = wl.fresh(r, np.arange(u.position, u.position + u.n_tokens))
        for pi, page in enumerate(u.pool_pages):
            j = np.arange(pi * B, min(u.n_tokens, (pi + 1) * B))
            kp, vp, ks, vs, filled = pages[int(page)]
            n = len(j)
            # pool page layout [H][B][d]: valid slots 0..n-1
            _check_nearest(e4m3_decode(kp[:, :n]).transpose(1, 0, 2) * ks, k[j], ks)
            _check_nearest(e4m3_decode(vp[:, :n]).transpose(1, 0, 2) * vs, v[j], vs)


def check_retained_tail_unfilled(wl):
    pages = C.retained_pages_e4m3(wl)
    B = wl.model.page_size
    seen_partial = False
    for r, u in _retained_units(wl):
        for pi, page in enumerate(u.pool_pages):
            n = min(u.n_tokens, (pi + 1) * B) - pi * B
            kp, vp, _, _, filled = pages[int(page)]
            assert filled[:n].all() and not filled[n:].any()
            assert not kp[:, n:].any() and not vp[:, n:].any()
            seen_partial |= n < B
    assert seen_partial


def check_retained_regather_at_zero_keeps_codes(wl):
    """A retained page gathered at offset 0 (rotation by angle 0) re-quantizes
    to its own codes and scale: the stored scale is already minimal."""
    pages = C.retained_pages_e4m3(wl)
    theta = wl.model.rope_theta
    for page, (kp, _, ks, _, filled) in pages.items():
        n = int(filled.sum())
        x = C.dequantize(kp[:, :n].transpose(1, 0, 2), ks)
        codes, s = C.quantize_page(rope_fp32(x, np.zeros(n, int), theta))
        assert s == ks
        assert np.array_equal(e4m3_decode(codes), e4m3_decode(kp[:, :n].transpose(1, 0, 2)))


def check_queries_per_row_head(wl, r=0):
    cpos, qd = C.quantized_queries_e4m3(wl, r)
    q, _, _ = wl.fresh(r, cpos)
    x = rope_fp32(q, cpos, wl.model.rope_theta)          # rotation pinned in test_oracle_rope
    amax = np.abs(x).max(axis=-1)
    T, H, _ = x.shape
    sc = np.empty((T, H))
    for t in range(T):
        for h in range(H):
            a = float(amax[t, h])
            s = 2.0 ** np.ceil(np.log2(a / 448.0)) if a else 1.0
            if a and a / s > 448.0:
                s *= 2
            _check_scale_minimal(a, s)
            sc[t, h] = s
    _check_nearest(qd, x, sc[..., None])


def test_retained_scales_are_minimal_per_page():
    check_retained_scales_minimal(_retain_workload())


def test_retained_codes_are_nearest_to_pre_rope_states():
    check_retained_codes_nearest_pre_rope(_retain_workload())


def test_retained_tail_slots_stay_unfilled():
    check_retained_tail_unfilled(_retain_workload())


def test_retained_unit_regathered_at_zero_keeps_its_codes():
    check_retained_regather_at_zero_keeps_codes(_retain_workload())


def test_queries_quantized_per_row_and_head():
    wl = workloads.generate("small_fp8")
    for r in range(len(wl.requests)):
        check_queries_per_row_head(wl, r)


def test_generator_pages_have_minimal_scales_at_varied_elements():
    """Every generated e4m3 pool page holds a +-448 code, so its scale is the
    minimal one, and that code is not always at the same element."""
    wl = workloads.generate("small_fp8")
    B = wl.model.page_size
    where = set()
    for uid in wl.hit_unit_ids():
        kc, vc, ks, vs = wl.unit_state_e4m3(uid)
        for codes, sc in ((kc, ks), (vc, vs)):
            for pi in range(len(sc)):
                pg = e4m3_decode(codes[pi * B:(pi + 1) * B])
                assert np.abs(pg).max() == 448.0
                _check_scale_minimal(float(np.abs(pg * sc[pi]).max()), sc[pi])
                where.add(tuple(np.argwhere(np.abs(pg) == 448.0)[0]))
    assert len(where) > 4


# ------------------------------------------------------- planted mistakes

def _retain_variant(rotate=False, unit_scale=False, scale_mul=1.0):
    """retained_pages_e4m3 with one deliberate mistake."""
    from oracle.numerics import e4m3_encode

    def f(wl):
        m = wl.model
        B = m.page_size
        out = {}
        for r, req in enumerate(wl.requests):
            for u in req.units:
                if u.residency != L.MISS or not u.retain:
                    continue
                pos = np.arange(u.position, u.position + u.n_tokens)
                _, k, v = wl.fresh(r, pos)
                if rotate:
                    k = rope_fp32(k, pos, m.rope_theta)
                for pi, page in enumerate(u.pool_pages):
                    j = np.arange(pi * B, min(u.n_tokens, (pi + 1) * B))
                    res = []
                    for x in (k, v):
                        src = x if unit_scale else x[j]
                        _, s = C.quantize_page(src)
                        s = np.float32(s * scale_mul)
                        res.append((e4m3_encode(x[j] / s), s))
                    (kc, ksc), (vc, vsc) = res
                    kp = np.zeros((m.n_kv_heads, B, m.head_dim), np.uint8)
                    vp = np.zeros_like(kp)
                    filled = np.zeros(B, dtype=bool)
                    kp[:, :len(j)] = kc.transpose(1, 0, 2)
                    vp[:, :len(j)] = vc.transpose(1, 0, 2)
                    filled[:len(j)] = True
                    out[int(page)] = (kp, vp, ksc, vsc, filled)
        return out
    return f


def _query_variant(per_row=False, unrotated=False):
    def f(wl, r, q_heads=None):
        from oracle.numerics import e4m3_encode, e4m3_page_scale
        cpos = L.compute_positions(wl.requests[r])
        q, _, _ = wl.fresh(r, cpos)
        qr = q if unrotated else rope_fp32(q, cpos, wl.model.rope_theta)
        amax = np.abs(qr).max(axis=(-1, -2) if per_row else -1)
        sc = e4m3_page_scale(amax.ravel()).reshape(amax.shape)
        sc = sc[:, None, None] if per_row else sc[..., None]
        return cpos, e4m3_decode(e4m3_encode(qr / sc)) * sc
    return f


@pytest.mark.parametrize("kw,check", [
    (dict(rotate=True), check_retained_codes_nearest_pre_rope),
    (dict(unit_scale=True), check_retained_scales_minimal),
    (dict(scale_mul=2.0), check_retained_scales_minimal),
])
def test_retention_mistakes_caught(monkeypatch, kw, check):
    wl = _retain_workload()
    monkeypatch.setattr(C, "retained_pages_e4m3", _retain_variant(**kw))
    with pytest.raises(AssertionError):
        check(wl)


@pytest.mark.parametrize("kw", [dict(per_row=True), dict(unrotated=True)])
def test_query_quantization_mistakes_caught(monkeypatch, kw):
    wl = workloads.generate("small_fp8")
    monkeypatch.setattr(C, "quantized_queries_e4m3", _query_variant(**kw))
    with pytest.raises(AssertionError):
        for r in range(len(wl.requests)):
            check_queries_per_row_head(wl, r)
