"""Pins for the composed path as a whole (oracle.pipeline)."""
from dataclasses import replace

import numpy as np
import pytest

import workloads
from oracle import layout as L
from oracle import pipeline as PL
from oracle.compose import assemble_request_kv


def _small(name="small_f32", **kw):
    cfg = workloads.get_config(name).with_(**kw)
    return workloads.make_workload(cfg)


def _all_recomputed(wl):
    for req in wl.requests:
        for u in req.units:
            u.n_recompute = u.n_tokens
    return wl


def _tie_units_to_fresh(wl):
    """Make every unit's cached pre-RoPE state equal the fresh projections of
    the tokens it covers (each unit id used once per batch)."""
    where = {}
    for r, req in enumerate(wl.requests):
        for u in req.units:
            where.setdefault(u.unit_id, (r, u.position, u.n_tokens))

    def state(uid):
        r, p, n = where[uid]
        _, k, v = wl.fresh(r, np.arange(p, p + n))
        return k, v
    wl.unit_state_fn = state
    return wl


@pytest.mark.parametrize("name", ["small_f32", "small_bf16"])
def test_every_token_recomputed_equals_full_prefill(name):
    wl = _all_recomputed(_small(name))
    for r, req in enumerate(wl.requests):
        res = PL.run_request(wl, r)
        assert len(res.positions) == req.prompt_len
        o, l = PL.full_prefill(wl, r)
        assert np.array_equal(res.out, o) and np.array_equal(res.lse, l)


def test_all_miss_equals_full_prefill():
    cfg = workloads.get_config("small_f32").with_(hit_prob=0.0)
    wl = workloads.make_workload(cfg)
    for r in range(len(wl.requests)):
        res = PL.run_request(wl, r)
        o, _ = PL.full_prefill(wl, r)
        assert np.array_equal(res.out, o)


@pytest.mark.parametrize("hit_prob,r", [(1.0, 0), (0.5, 3), (1.0, 200)])
def test_output_invariant_to_residency_when_cache_matches_fresh(hit_prob, r):
    """If the pool holds exactly the pre-RoPE states the request would compute,
    composing them changes nothing: same assembled KV, same outputs (exact,
    since both routes rotate with the same fp32 evaluation)."""
    cfg = workloads.get_config("small_f32").with_(
        hit_prob=hit_prob, n_recompute=r, unit_order=((0, 1, 2), (3, 4, 5)),
        units_per_request=3)
    wl = _tie_units_to_fresh(workloads.make_workload(cfg))
    ref = _all_recomputed(_tie_units_to_fresh(workloads.make_workload(cfg)))
    for q in range(2):
        a = PL.run_request(wl, q)
        b = PL.run_request(ref, q)
        assert np.array_equal(a.K, b.K) and np.array_equal(a.V, b.V)
        common = np.isin(b.positions, a.positions)
        idx = np.searchsorted(b.positions, a.positions)
        assert np.array_equal(a.out, b.out[idx])
        assert common.sum() == len(a.positions)


def test_values_are_copied_and_keys_rotated():
    wl = _small("small_bf16")
    for r, req in enumerate(wl.requests):
        K, V, src = assemble_request_kv(wl, r)
        assert not np.isnan(K).any() and not np.isnan(V).any()
        for u in req.units:
            if u.residency != L.HIT or u.n_recompute >= u.n_tokens:
                continue
            k_pre, v = wl.unit_state(u.unit_id)
            j0 = u.n_recompute
            assert np.array_equal(V[u.position + j0:u.position + u.n_tokens], v[j0:])
            assert not np.array_equal(K[u.position + j0:u.position + u.n_tokens], k_pre[j0:])


def test_tiny_counts_follow_config():
    wl = workloads.generate("tiny")
    c = PL.counts(wl)
    # [M,H,M,H] x 64 tokens + 16 query, r = 4: 2*64 + 2*4 + 16 computed
    assert c["compute_tokens"] == 152 and c["gather_tokens"] == 120
    assert c["prompt_tokens"] == 272


def test_retained_pages_are_prerope_fresh_values():
    wl = _small("small_f32")
    pages = PL.retained_pages(wl) if hasattr(PL, "retained_pages") else None
    from oracle.compose import retained_pages
    pages = retained_pages(wl)
    assert pages
    B = wl.model.page_size
    for r, req in enumerate(wl.requests):
        for u in req.units:
            if u.residency == L.MISS and u.retain:
                _, k, v = wl.fresh(r, np.arange(u.position, u.position + u.n_tokens))
                for j in range(u.n_tokens):
                    pk, pv, filled = pages[int(u.pool_pages[j // B])]
                    assert filled[j % B]
                    assert np.array_equal(pk[:, j % B], k[j])
                    assert np.array_equal(pv[:, j % B], v[j])
                last = pages[int(u.pool_pages[-1])][2]
                tail = u.n_tokens % B
                if tail:
                    assert not last[tail:].any()
