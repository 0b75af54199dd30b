"""Pins for the LOCAL miss scope of the oracle (Section 5.3: missing units
are prefilled independently, then composed like hits with a recompute
window)."""
import numpy as np
import pytest

import workloads
from oracle import attention as A
from oracle import layout as L
from oracle import pipeline as PL


def _wl(name="tiny", **kw):
    return workloads.make_workload(workloads.get_config(name).with_(**kw))


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def test_row_kv_lo_by_hand():
    """Tiny, pattern [MISS, HIT, MISS, HIT], r = 4, units of 64 at 0, 64, 128,
    192, query at 256: the MISS units' tokens past their window see only
    their own unit; windows and the query see everything."""
    wl = _wl(miss_scope="local", residency_pattern=(0, 1, 0, 1))
    req = wl.requests[0]
    pos = L.compute_positions(req)
    lo = L.row_kv_lo(req)
    want = np.zeros(len(pos), dtype=np.int64)
    for start in (0, 128):                      # the two MISS units
        sel = (pos >= start + 4) & (pos < start + 64)
        want[sel] = start
    assert np.array_equal(lo, want)
    assert int(((pos >= 4) & (pos < 64)).sum()) == 60
    # GLOBAL scope: every row sees the whole prefix
    assert not L.row_kv_lo(_wl(residency_pattern=(0, 1, 0, 1)).requests[0]).any()


def test_attention_with_kv_lo_matches_brute_force():
    rng = np.random.default_rng(7)
    T, Hq, Hkv, d, P = 6, 4, 2, 4, 9
    q = rng.standard_normal((T, Hq, d))
    K = rng.standard_normal((P, Hkv, d))
    V = rng.standard_normal((P, Hkv, d))
    pos = np.array([0, 2, 3, 5, 7, 8])
    lo = np.array([0, 1, 3, 2, 7, 0])
    o, s = A.causal_gqa_attention(q, pos, K, V, kv_lo=lo)
    ob, sb = A.brute_force_attention(q.tolist(), pos, K.tolist(), V.tolist(), kv_lo=lo)
    assert np.allclose(o, ob, rtol=1e-12, atol=1e-12)
    assert np.allclose(s, sb, rtol=1e-12, atol=1e-12)
    # a row whose window is one key returns that key's value exactly
    assert np.array_equal(o[4], np.repeat(V[7], Hq // Hkv, axis=0))


@pytest.mark.parametrize("pattern", [(1, 1, 1, 1), (0, 1, 0, 1)])
def test_local_equals_global_when_no_miss_row_is_unit_local(pattern):
    """All hits, or every miss token inside its window: nothing changes."""
    kw = dict(residency_pattern=pattern)
    if 0 in pattern:
        kw["n_recompute"] = 64                  # windows cover whole units
    g = PL.run_request(_wl(**kw), 0)
    l = PL.run_request(_wl(miss_scope="local", **kw), 0)
    assert not l.kv_lo.any()
    assert np.array_equal(g.out, l.out) and np.array_equal(g.lse, l.lse)


@pytest.mark.parametrize("name", ["tiny", "small_f32"])
def test_local_miss_rows_equal_independent_prefill(name):
    """A MISS unit's rows past its window equal the unit prefilled alone from
    position 0 (RoPE relativity; fp32 rotation rounding only)."""
    wl = _wl(name, miss_scope="local")
    checked = 0
    for r, req in enumerate(wl.requests):
        res = PL.run_request(wl, r)
        row_of = {int(p): i for i, p in enumerate(res.positions)}
        for ui, u in enumerate(req.units):
            if u.residency != L.MISS:
                continue
            rwin = min(int(u.n_recompute), int(u.n_tokens))
            if rwin >= u.n_tokens:
                continue
            alone, _ = PL.unit_prefill(wl, r, ui)
            rows = [row_of[u.position + j] for j in range(rwin, u.n_tokens)]
            got = res.out[rows]
            want = alone[rwin:][:, res.q_heads]
            assert _rel(got, want) < 2e-5, (r, ui, _rel(got, want))
            checked += 1
    assert checked > 0


def test_a_shifted_window_start_is_caught(monkeypatch):
    """Planted mistake: unit-local rows starting one key late."""
    wl = _wl("tiny", miss_scope="local")
    orig = L.row_kv_lo

    def late(req):
        lo = orig(req)
        return np.where(lo > 0, lo + 1, lo)
    monkeypatch.setattr(L, "row_kv_lo", late)
    res = PL.run_request(wl, 0)
    u = wl.requests[0].units[2]                 # MISS unit at 128
    rwin = min(u.n_recompute, u.n_tokens)
    alone, _ = PL.unit_prefill(wl, 0, 2)
    row_of = {int(p): i for i, p in enumerate(res.positions)}
    rows = [row_of[u.position + j] for j in range(rwin, u.n_tokens)]
    assert _rel(res.out[rows], alone[rwin:]) > 1e-3


def test_local_visible_pairs():
    """LOCAL keeps the computed rows and shrinks the attention work by the
    keys before every unit-local row's unit."""
    for name in ("tiny", "rag8b"):
        cfg = workloads.get_config(name)
        g = PL.counts(workloads.make_workload(cfg))
        l = PL.counts(workloads.make_workload(cfg.with_(miss_scope="local")))
        assert g["compute_tokens"] == l["compute_tokens"]
        assert g["gather_tokens"] == l["gather_tokens"]
        assert l["visible_pairs"] < g["visible_pairs"]
    wl = _wl(miss_scope="local")
    req = wl.requests[0]
    pos, lo = L.compute_positions(req), L.row_kv_lo(req)
    assert PL.counts(wl)["visible_pairs"] == int((pos - lo + 1).sum())
