"""Retrieval-aware caching and routing, written out plainly (Section 5.2).
TEST INFRASTRUCTURE ONLY.

Everything is recomputed from the request history on every call: the score
recounts the retrieval history, admission sorts every resident unit, and
routing scans every node.  Nothing is cached or incrementally maintained.

* score            -- s(u,t) = w_r f_W(u,t) + w_l f_inf(u,t) (the reuse
                      estimate of Section 5.2).
* window_for_capacity -- W, the number of requests whose retrieved units
                      fill the cache.
* admit            -- threshold admission; eviction of strictly lower-scored
                      whole units, capacity counted in blocks.
* route            -- least-loaded-within-one, then most local blocks, then
                      lower load, then round-robin.
* replay           -- the trace replay the library implements.

Readings (where Section 5.2 is silent):
* The request being served is part of the history its own admission
  decision sees (t counts it), so a unit's first retrieval scores
  w_r + w_l = 1.05, below the default threshold.
* theta defaults to 2.0: admission needs a second retrieval within the
  window, or a long lifetime count, and never the first retrieval alone.
* Units with equal scores are considered in increasing unit id.
* A request lists a unit at most once; a repeat is ignored.
* W = floor(capacity_blocks / mean blocks per request), at least 1.
* The replay keeps a request in flight until `concurrency` later requests
  have arrived; admissions of one request follow its retrieval order.

Parity: pinned by tests/test_control_plane.py with hand-worked traces of
each rule; the library is compared with these functions on random traces.
"""
from __future__ import annotations

import math

BELOW_THRESHOLD, ADMITTED, RESIDENT, NO_ROOM, TOO_LARGE = range(5)


def dedupe(units):
    seen, out = set(), []
    for u in units:
        if u not in seen:
            seen.add(u)
            out.append(u)
    return out


def score(history, unit, window, w_recent=1.0, w_lifetime=0.05):
    """history: the request stream so far (lists of unit ids), oldest first."""
    recent = sum(1 for req in history[-window:] if unit in req) if window > 0 else 0
    lifetime = sum(1 for req in history if unit in req)
    return w_recent * recent + w_lifetime * lifetime


def window_for_capacity(capacity_blocks, mean_blocks_per_request):
    if mean_blocks_per_request <= 0 or capacity_blocks <= 0:
        return 1
    return max(1, math.floor(capacity_blocks / mean_blocks_per_request))


def admit(resident, capacity, theta, history, window, unit, n_blocks,
          w_recent=1.0, w_lifetime=0.05):
    """resident: dict unit -> blocks (modified when admitted).
    Returns (result, victims)."""
    if unit in resident:
        return RESIDENT, []
    s = score(history, unit, window, w_recent, w_lifetime)
    if s < theta:
        return BELOW_THRESHOLD, []
    if n_blocks > capacity:
        return TOO_LARGE, []
    free = capacity - sum(resident.values())
    victims = []
    if free < n_blocks:
        ranked = sorted((score(history, v, window, w_recent, w_lifetime), v) for v in resident)
        for sv, v in ranked:
            if free >= n_blocks or not sv < s:
                break
            victims.append(v)
            free += resident[v]
        if free < n_blocks:
            return NO_ROOM, []
    for v in victims:
        del resident[v]
    resident[unit] = n_blocks
    return ADMITTED, victims


def route(node_resident, inflight, units, rr):
    """node_resident: per node, dict unit -> blocks (or None).  Returns
    (node, next cursor)."""
    n = len(inflight)
    least = min(inflight)
    units = dedupe(units)
    best = None
    for k in range(n):
        i = (rr + k) % n
        if inflight[i] > least + 1:
            continue
        res = node_resident[i] or {}
        blocks = sum(res.get(u, 0) for u in units)
        key = (blocks, -inflight[i])
        if best is None or key > best[0]:
            best = (key, i)
    return best[1], (best[1] + 1) % n


def replay(requests, n_nodes, local_capacity, shared_capacity, page_size, theta=2.0,
           w_recent=1.0, w_lifetime=0.05, local_window=0, shared_window=0, concurrency=8,
           cache_aware=True):
    """requests: list of (unit ids, unit token counts).  Returns (stats, routes)."""
    reqs = [dedupe(ids) for ids, _ in requests]
    length = {}
    for ids, toks in requests:
        for u, t in zip(ids, toks):
            length[u] = t
    blocks = {u: -(-t // page_size) for u, t in length.items()}
    mean = (sum(blocks[u] for r in reqs for u in r) / len(reqs)) if reqs else 1.0
    wl = local_window or window_for_capacity(local_capacity, mean)
    ws = shared_window or window_for_capacity(shared_capacity, mean)
    local = [dict() for _ in range(n_nodes)]
    local_hist = [[] for _ in range(n_nodes)]
    shared, shared_hist = {}, []
    has_shared = shared_capacity > 0
    inflight = [0] * n_nodes
    flying = []
    per_node = [0] * n_nodes
    rr = 0
    st = dict.fromkeys(["requests", "unit_refs", "blocks", "local_hit_units", "local_hit_blocks",
                        "shared_hit_units", "shared_hit_blocks", "miss_units", "miss_blocks",
                        "local_admitted", "local_evicted", "shared_admitted",
                        "shared_evicted", "max_node_requests", "min_node_requests"], 0)
    routes = []
    for units in reqs:
        node, rr = route(local if cache_aware else [None] * n_nodes, inflight, units, rr)
        routes.append(node)
        per_node[node] += 1
        inflight[node] += 1
        flying.append(node)
        if len(flying) > concurrency:
            inflight[flying.pop(0)] -= 1
        in_local = [u in local[node] for u in units]
        in_shared = [has_shared and u in shared for u in units]
        for u, a, b in zip(units, in_local, in_shared):
            st["unit_refs"] += 1
            st["blocks"] += blocks[u]
            tier = "local" if a else "shared" if b else "miss"
            key = "miss" if tier == "miss" else f"{tier}_hit"
            st[f"{key}_units"] += 1
            st[f"{key}_blocks"] += blocks[u]
        local_hist[node].append(set(units))
        if has_shared:
            shared_hist.append(set(units))
        for u, a, b in zip(units, in_local, in_shared):
            if not a:
                r, v = admit(local[node], local_capacity, theta, local_hist[node], wl, u,
                             blocks[u], w_recent, w_lifetime)
                if r == ADMITTED:
                    st["local_admitted"] += 1
                    st["local_evicted"] += len(v)
            if has_shared and not b:
                r, v = admit(shared, shared_capacity, theta, shared_hist, ws, u, blocks[u],
                             w_recent, w_lifetime)
                if r == ADMITTED:
                    st["shared_admitted"] += 1
                    st["shared_evicted"] += len(v)
    st["requests"] = len(reqs)
    st["max_node_requests"] = max(per_node) if reqs else 0
    st["min_node_requests"] = min(per_node) if reqs else 0
    return st, routes
