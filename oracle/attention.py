"""Causal GQA prefill attention over the assembled KV (oracle).

Follows Section 5.3 "Completing prefill": the tokens selected for
recomputation and the remaining prompt are processed in one extend pass whose
attention sees the request's whole assembled KV up to each token's position.
Definition used (readings for what the paper leaves unstated):

* query head h uses KV head g = floor(h / G), G = H_q / H_kv (contiguous
  grouping, as in Llama-family GQA);
* a token at prompt position p sees keys at positions lo .. p inclusive,
  lo = 0 except for the unit-local rows of LOCAL miss scope (layout.py);
* s_j = scale * <q, k_j>, scale = 1/sqrt(d) unless given;
* o = sum_j softmax(s)_j v_j, lse = logsumexp(s) (natural log);
* everything in fp64, on operands already rounded to the dtypes the GPU
  consumes.

Pins (tests/test_oracle_attention.py): brute-force pure-Python loops on tiny
inputs; torch's CPU scaled_dot_product_attention in float64 with an explicit
boolean mask and repeated KV heads; one visible key gives o = v exactly;
q = 0 gives the mean of the visible values; softmax rows sum to one.
"""
from __future__ import annotations

import math

import numpy as np


def causal_gqa_attention(q, positions, K, V, scale=None, row_block: int = 1024,
                         kv_lo=None):
    """q [T][H_q][d], positions [T], K/V [P][H_kv][d] -> out [T][H_q][d], lse [T][H_q].

    kv_lo [T] (optional): first visible key of every row (default 0).

    All arithmetic in fp64.  Rows are evaluated in blocks of `row_block`
    only to bound memory; every row is independent.
    """
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    positions = np.asarray(positions, dtype=np.int64)
    T, Hq, d = q.shape
    Hkv = K.shape[1]
    if Hq % Hkv:
        raise ValueError("H_q must be a multiple of H_kv")
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = np.zeros((T, Hq, d), dtype=np.float64)
    lse = np.zeros((T, Hq), dtype=np.float64)
    if T == 0:
        return out, lse
    lo_all = (np.zeros(T, dtype=np.int64) if kv_lo is None
              else np.asarray(kv_lo, dtype=np.int64))
    P = int(positions.max()) + 1
    key_pos = np.arange(P)
    for r0 in range(0, T, row_block):
        rows = slice(r0, min(T, r0 + row_block))
        pr = positions[rows]
        visible = ((key_pos[None, :] <= pr[:, None]) &
                   (key_pos[None, :] >= lo_all[rows][:, None]))   # [t][P]
        for h in range(Hq):
            g = h // G
            s = scale * (q[rows, h, :] @ K[:P, g, :].T)      # [t][P]
            s = np.where(visible, s, -np.inf)
            mx = s.max(axis=1, keepdims=True)
            e = np.exp(s - mx)
            l = e.sum(axis=1, keepdims=True)
            out[rows, h, :] = (e @ V[:P, g, :]) / l
            lse[rows, h] = (mx + np.log(l))[:, 0]
    return out, lse


def brute_force_attention(q, positions, K, V, scale=None, kv_lo=None):
    """Same definition with explicit Python loops (tiny inputs only)."""
    T, Hq, d = len(q), len(q[0]), len(q[0][0])
    Hkv = len(K[0])
    G = Hq // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = [[[0.0] * d for _ in range(Hq)] for _ in range(T)]
    lse = [[0.0] * Hq for _ in range(T)]
    for t in range(T):
        p = int(positions[t])
        lo = 0 if kv_lo is None else int(kv_lo[t])
        keys = list(range(lo, p + 1))
        for h in range(Hq):
            g = h // G
            scores = []
            for j in keys:
                acc = 0.0
                for c in range(d):
                    acc += float(q[t][h][c]) * float(K[j][g][c])
                scores.append(scale * acc)
            mx = max(scores)
            w = [math.exp(s - mx) for s in scores]
            tot = sum(w)
            for c in range(d):
                out[t][h][c] = sum(w[i] * float(V[j][g][c]) for i, j in enumerate(keys)) / tot
            lse[t][h] = mx + math.log(tot)
    return np.array(out), np.array(lse)
