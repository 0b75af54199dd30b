"""Pins for the oracle's e4m3 pool path (a reading: the paper has no 8-bit
path).  Built on oracle.numerics, which is pinned to torch's casts."""
from types import SimpleNamespace as NS

import numpy as np
import pytest

import workloads
from oracle import compose as C
from oracle import layout as L
from oracle import pipeline as PL
from oracle.numerics import e4m3_decode


def test_quantize_page_roundtrip_and_scale():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((16, 8, 128)).astype(np.float32) * 3
    codes, s = C.quantize_page(x)
    amax = np.abs(x).max()
    assert amax / s <= 448 and amax / (s / 2) > 448
    y = C.dequantize(codes, s)
    # nearest-even rounding: error at most half a quantum of each binade
    assert np.all(np.abs(y - x) <= np.abs(x) * 2.0**-4 + s * 2.0**-10)
    # values already on the grid survive a second quantization unchanged
    c2, s2 = C.quantize_page(y)
    assert s2 == s and np.array_equal(c2, codes)


def test_zero_page_has_unit_scale():
    codes, s = C.quantize_page(np.zeros((3, 2, 4), np.float32))
    assert s == 1.0 and not codes.any()


def test_unrotated_page_requantizes_to_its_own_codes():
    """Dequantize -> rotate at position 0 (the identity) -> requantize returns
    a stored page unchanged: its scale is already the minimal one."""
    wl = workloads.generate("small_fp8")
    B = wl.model.page_size
    for uid in wl.hit_unit_ids()[:4]:
        kc, vc, kscale, vscale = wl.unit_state_e4m3(uid)
        for pi in range(len(kscale)):
            j = np.arange(pi * B, min(len(kc), (pi + 1) * B))
            x = C.rope_fp32(C.dequantize(kc[j], kscale[pi]), np.zeros(len(j), int),
                            wl.model.rope_theta)
            codes, s = C.quantize_page(x)
            # compare values: rotation may turn -0.0 into +0.0 (IEEE rules)
            assert s == kscale[pi]
            assert np.array_equal(e4m3_decode(codes), e4m3_decode(kc[j]))


def test_gathered_values_are_copied_with_their_scales():
    cfg = workloads.get_config("small_fp8").with_(
        instruction_tokens=0, hit_prob=1.0, n_recompute=0, unit_order=((3, 1, 2),),
        n_requests=1, units_per_request=3)
    wl = workloads.make_workload(cfg)
    Kc, Vc, ks, vs = C.assemble_request_kv_e4m3(wl, 0)
    B = wl.model.page_size
    for u in wl.requests[0].units:
        kc, vc, kscale, vscale = wl.unit_state_e4m3(u.unit_id)
        sl = slice(u.position, u.position + u.n_tokens)
        assert np.array_equal(Vc[sl], vc)
        assert np.array_equal(vs[sl], np.repeat(vscale, B)[:u.n_tokens])
        assert not np.array_equal(Kc[sl], kc)       # keys are re-rotated


def test_rerotated_keys_match_fp32_rotation_within_quantization():
    wl = workloads.generate("small_fp8")
    for r, req in enumerate(wl.requests):
        Kc, _, ks, _ = C.assemble_request_kv_e4m3(wl, r)
        for u in req.units:
            if u.residency != L.HIT or L.recompute_count(u) >= u.n_tokens:
                continue
            kc, _, kscale, _ = wl.unit_state_e4m3(u.unit_id)
            j = np.arange(L.recompute_count(u), u.n_tokens)
            pos = u.position + j
            B = wl.model.page_size
            exact = C.rope_fp32(e4m3_decode(kc[j]) * np.repeat(kscale, B)[j][:, None, None],
                                pos, wl.model.rope_theta)
            got = e4m3_decode(Kc[pos]) * ks[pos][:, None, None]
            tol = np.abs(exact) * 2.0**-4 + ks[pos][:, None, None] * 2.0**-9
            assert np.all(np.abs(got - exact) <= tol)


def test_misaligned_plans_are_rejected():
    req = NS(prompt_len=40, text_segs=[(0, 8)],
             units=[NS(unit_id=0, position=8, n_tokens=32, residency=L.HIT,
                       n_recompute=0, retain=0, pool_pages=np.arange(2))])
    with pytest.raises(ValueError):
        C.check_page_aligned(req, 16)


def test_fp8_attention_runs_on_dequantized_operands():
    wl = workloads.generate("small_fp8")
    res = PL.run_request(wl, 0, kv_heads=[1])
    assert np.isfinite(res.out).all() and res.out.shape[1] == 4
    # queries are on the per-row e4m3 grid
    q = res.q
    amax = np.abs(q).max(axis=-1, keepdims=True)
    s = 2.0 ** np.ceil(np.log2(amax / 448))
    assert np.array_equal(e4m3_decode(np.zeros(1, np.uint8)), [0.0])
    assert np.all(np.abs(q / s) <= 448)
