"""The control plane (Section 5.2): the oracle pinned by hand-worked cases of
each rule, then the library compared with the oracle on random traces."""
import ctypes

import numpy as np
import pytest

import paper_2609_32999_amd._binding as B
from oracle import control as C
from workloads.traces import zipf_trace


# ------------------------------------------------------------ oracle pins
def test_score_counts_recent_window_and_lifetime():
    h = [{1, 2}, {2}, {3}, {2, 1}]
    # last two requests: {3}, {1, 2}
    assert C.score(h, 2, window=2) == pytest.approx(1 + 0.05 * 3)
    assert C.score(h, 1, window=2) == pytest.approx(1 + 0.05 * 2)
    assert C.score(h, 3, window=2) == pytest.approx(1 + 0.05 * 1)
    assert C.score(h, 2, window=4) == pytest.approx(3 + 0.05 * 3)
    assert C.score(h, 9, window=4) == 0.0


def test_first_retrieval_is_not_admitted_second_is():
    res, hist = {}, [{7}]
    assert C.admit(res, 100, 2.0, hist, 4, 7, 3) == (C.BELOW_THRESHOLD, [])
    hist.append({7})
    assert C.admit(res, 100, 2.0, hist, 4, 7, 3) == (C.ADMITTED, [])
    assert res == {7: 3}
    assert C.admit(res, 100, 2.0, hist, 4, 7, 3) == (C.RESIDENT, [])


def test_eviction_takes_only_strictly_lower_scores_lowest_first():
    hist = [{1}, {1}, {2}, {2}, {2}, {3}, {3}]        # window 7
    res = {1: 4, 2: 4}                                # scores 2.1, 3.15; cap 8, full
    # unit 3 scores 2.1: ties unit 1, beats nothing strictly -> no room
    assert C.admit(dict(res), 8, 2.0, hist, 7, 3, 4) == (C.NO_ROOM, [])
    hist.append({3})                                  # unit 3 -> 3.15: beats unit 1 only
    r = dict(res)
    assert C.admit(r, 8, 2.0, hist, 8, 3, 4) == (C.ADMITTED, [1])
    assert r == {2: 4, 3: 4}
    # needing 8 blocks it would also need unit 2, which ties -> no room
    assert C.admit(dict(res), 8, 2.0, hist, 8, 3, 8)[0] == C.NO_ROOM
    assert C.admit({}, 8, 2.0, hist, 8, 3, 9) == (C.TOO_LARGE, [])


def test_fading_demand_is_displaced():
    W = 3
    hist = [{1}, {1}, {1}]                            # unit 1: 3.15
    res = {}
    assert C.admit(res, 4, 2.0, hist, W, 1, 4)[0] == C.ADMITTED
    hist += [{2}, {2}]                                # unit 1 falls out of the window
    assert C.score(hist, 1, W) == pytest.approx(1 + 0.15)
    assert C.admit(res, 4, 2.0, hist, W, 2, 4) == (C.ADMITTED, [1])


def test_route_load_window_blocks_then_load_then_round_robin():
    a, b, c = {10: 5}, {10: 5, 11: 2}, {}
    # node 1 holds most blocks but is 2 above the least loaded: excluded
    assert C.route([a, b, c], [1, 3, 1], [10, 11], 0)[0] == 0
    # within one of the least loaded: the most blocks wins
    assert C.route([a, b, c], [1, 2, 1], [10, 11], 0)[0] == 1
    # equal blocks: lower load
    assert C.route([a, dict(a), c], [2, 1, 1], [10], 0)[0] == 1
    # all equal: round-robin from the cursor
    n, rr = C.route([c, c, c], [0, 0, 0], [5], 0)
    n2, rr = C.route([c, c, c], [0, 0, 0], [5], rr)
    n3, rr = C.route([c, c, c], [0, 0, 0], [5], rr)
    assert (n, n2, n3) == (0, 1, 2) and rr == 0


def test_window_fills_the_cache():
    assert C.window_for_capacity(100, 30.0) == 3
    assert C.window_for_capacity(10, 30.0) == 1
    assert C.window_for_capacity(0, 30.0) == 1


def test_replay_small_trace_by_hand():
    # one node, capacity 4 blocks, B = 16, theta 2, W 8
    trace = [([1], [32]), ([1], [32]), ([1], [32]), ([2], [64]), ([1, 2], [32, 64])]
    st, routes = C.replay(trace, 1, 4, 0, 16, local_window=8, concurrency=1)
    # r0: miss, 1 -> 1.05 no.  r1: miss, 1 -> 2.1 admitted (2 blocks).
    # r2: hit.  r3: miss 2 (1.05).  r4: hit 1; 2 -> 2.1 needs 4 blocks, 2
    # free; unit 1 scores 4.25 -> no room
    assert st["local_hit_units"] == 2 and st["miss_units"] == 4
    assert st["local_admitted"] == 1 and st["local_evicted"] == 0
    assert st["blocks"] == 2 * 4 + 4 + 4 and routes == [0] * 5


# -------------------------------------------------- library against oracle
def test_library_scorer_matches_oracle():
    rng = np.random.default_rng(1)
    for window in (1, 3, 17):
        s = B.Scorer(window)
        hist = []
        for _ in range(200):
            req = list(rng.integers(0, 30, size=rng.integers(0, 8)))
            s.observe(req)
            hist.append(set(req))
            for u in range(30):
                assert s.score(u) == C.score(hist, u, window), (window, u)
        r, l = s.counts(3)
        assert l == sum(3 in h for h in hist) and r == sum(3 in h for h in hist[-window:])


def test_library_admission_matches_oracle():
    rng = np.random.default_rng(2)
    for cap, theta, window in ((40, 2.0, 6), (12, 1.5, 3), (100, 3.0, 20)):
        s = B.Scorer(window)
        a = B.Admitter(cap, theta)
        hist, res = [], {}
        for _ in range(400):
            req = [int(x) for x in rng.zipf(1.3, size=4) % 50]
            s.observe(req)
            hist.append(set(req))
            for u in C.dedupe(req):
                nb = 1 + u % 7
                got = a.admit(s, u, nb)
                want = C.admit(res, cap, theta, hist, window, u, nb)
                assert got == (want[0], want[1]), (u, got, want)
            assert a.used_blocks == sum(res.values()) and a.num_units == len(res)
        for u, nb in res.items():
            assert a.blocks(u) == nb


def test_library_admission_victim_overflow_changes_nothing():
    s = B.Scorer(8)
    a = B.Admitter(4, 0.5)
    for u in range(4):
        s.observe([u])
        assert a.admit(s, u, 1)[0] == B.TSR_ADMIT_ADMITTED
    s.observe([9])
    s.observe([9])
    with pytest.raises(B.TsrError) as e:
        a.admit(s, 9, 4, max_victims=2)
    assert e.value.status == B.TSR_ERR_OUT_OF_RANGE
    assert a.num_units == 4 and a.used_blocks == 4
    assert a.admit(s, 9, 4)[1] == [0, 1, 2, 3]


def test_library_route_matches_oracle():
    rng = np.random.default_rng(3)
    for _ in range(300):
        n = int(rng.integers(1, 6))
        caches, dicts = [], []
        s = B.Scorer(4)
        for i in range(n):
            a = B.Admitter(1000, 0.0)
            d = {}
            for u in rng.choice(20, size=rng.integers(0, 8), replace=False):
                nb = int(1 + u % 5)
                s.observe([int(u)])
                a.admit(s, int(u), nb)
                d[int(u)] = nb
            caches.append(a)
            dicts.append(d)
        inflight = list(rng.integers(0, 4, size=n))
        units = [int(x) for x in rng.integers(0, 20, size=rng.integers(0, 6))]
        rr = int(rng.integers(0, n))
        assert B.tsr_route(caches, inflight, units, rr) == C.route(dicts, inflight, units, rr)


def _cfg(**kw):
    base = dict(n_nodes=4, local_capacity_blocks=400, shared_capacity_blocks=0, page_size=16,
                theta=2.0, w_recent=1.0, w_lifetime=0.05, local_window=0, shared_window=0,
                concurrency=8, cache_aware=1)
    base.update(kw)
    return B.tsr_replay_config(**base)


@pytest.mark.parametrize("kw", [
    {}, {"n_nodes": 1}, {"shared_capacity_blocks": 900}, {"cache_aware": 0},
    {"n_nodes": 3, "local_capacity_blocks": 150, "concurrency": 2},
    {"theta": 1.0, "local_window": 5, "shared_capacity_blocks": 300, "shared_window": 9},
])
def test_library_replay_matches_oracle(kw):
    trace = zipf_trace(5, 300, 400, 6, zipf_s=1.1, token_range=(20, 200), drift_every=100,
                       drift_shift=37)
    cfg = _cfg(**kw)
    st, routes = B.tsr_replay(cfg, trace, return_routes=True)
    want, wroutes = C.replay([([int(u) for u in i], [int(t) for t in k]) for i, k in trace],
                             cfg.n_nodes, cfg.local_capacity_blocks, cfg.shared_capacity_blocks,
                             cfg.page_size, cfg.theta, cfg.w_recent, cfg.w_lifetime,
                             cfg.local_window, cfg.shared_window, cfg.concurrency,
                             bool(cfg.cache_aware))
    assert st == want
    assert list(routes) == wroutes
    assert st["local_hit_units"] + st["shared_hit_units"] + st["miss_units"] == st["unit_refs"]
    assert st["local_hit_blocks"] + st["shared_hit_blocks"] + st["miss_blocks"] == st["blocks"]


def test_replay_rejects_changing_lengths_and_bad_config():
    with pytest.raises(B.TsrError):
        B.tsr_replay(_cfg(), [([1], [10]), ([1], [11])])
    with pytest.raises(B.TsrError):
        B.tsr_replay(_cfg(n_nodes=0), [([1], [10])])
    with pytest.raises(B.TsrError):
        B.tsr_replay(_cfg(concurrency=0), [([1], [10])])
