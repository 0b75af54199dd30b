"""Pins for oracle.attention (causal GQA prefill over the assembled KV)."""
import math

import numpy as np
import pytest
import torch

from oracle.attention import brute_force_attention, causal_gqa_attention


def _case(seed, T, P, Hq, Hkv, d, positions=None):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((T, Hq, d))
    K = rng.standard_normal((P, Hkv, d))
    V = rng.standard_normal((P, Hkv, d))
    if positions is None:
        positions = np.sort(rng.choice(P, size=T, replace=False))
    return q, np.asarray(positions), K, V


def test_matches_brute_force_loops():
    # 3 units x 5 tokens + 2 text tokens, d = 4, two query heads per KV head
    q, pos, K, V = _case(0, T=9, P=17, Hq=4, Hkv=2, d=4)
    o, l = causal_gqa_attention(q, pos, K, V)
    ob, lb = brute_force_attention(q.tolist(), pos, K.tolist(), V.tolist())
    assert np.allclose(o, ob, rtol=1e-12, atol=1e-12)
    assert np.allclose(l, lb, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 2), (8, 1)])
def test_matches_torch_sdpa_float64(Hq, Hkv):
    q, pos, K, V = _case(1, T=40, P=97, Hq=Hq, Hkv=Hkv, d=32)
    o, _ = causal_gqa_attention(q, pos, K, V)
    G = Hq // Hkv
    P = int(pos.max()) + 1
    qt = torch.from_numpy(q).permute(1, 0, 2)                        # [Hq][T][d]
    kt = torch.from_numpy(K[:P]).permute(1, 0, 2).repeat_interleave(G, 0)
    vt = torch.from_numpy(V[:P]).permute(1, 0, 2).repeat_interleave(G, 0)
    mask = torch.from_numpy(np.arange(P)[None, :] <= pos[:, None])   # [T][P]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask)
    assert np.allclose(o, ref.permute(1, 0, 2).numpy(), rtol=1e-11, atol=1e-12)


def test_single_visible_key_returns_its_value_exactly():
    q, _, K, V = _case(2, T=1, P=5, Hq=2, Hkv=1, d=8)
    o, l = causal_gqa_attention(q, np.array([0]), K, V)
    assert np.array_equal(o[0, 0], V[0, 0]) and np.array_equal(o[0, 1], V[0, 0])
    assert np.allclose(l[0], (q[0] @ K[0, 0]) / math.sqrt(8))


def test_zero_query_averages_visible_values():
    _, _, K, V = _case(3, T=3, P=50, Hq=2, Hkv=2, d=16)
    q = np.zeros((3, 2, 16))
    pos = np.array([0, 9, 49])
    o, l = causal_gqa_attention(q, pos, K, V)
    for t, p in enumerate(pos):
        assert np.allclose(o[t], V[:p + 1].mean(axis=0), rtol=1e-13, atol=1e-14)
        assert np.allclose(l[t], math.log(p + 1))


def test_softmax_rows_sum_to_one_via_lse():
    q, pos, K, V = _case(4, T=20, P=64, Hq=4, Hkv=2, d=16)
    _, lse = causal_gqa_attention(q, pos, K, V)
    for t in range(20):
        for h in range(4):
            s = (K[:pos[t] + 1, h // 2] @ q[t, h]) / 4.0
            assert abs(np.exp(s - lse[t, h]).sum() - 1.0) < 1e-13


def test_causality_future_keys_do_not_matter():
    q, pos, K, V = _case(5, T=6, P=30, Hq=2, Hkv=1, d=8, positions=[3, 4, 10, 11, 20, 21])
    o1, _ = causal_gqa_attention(q, pos, K, V)
    K2, V2 = K.copy(), V.copy()
    K2[22:] = 1e3
    V2[22:] = -1e3
    K2[11:21] += 0  # unchanged range
    o2, _ = causal_gqa_attention(q, pos, K2, V2)
    assert np.array_equal(o1, o2)
    # a key exactly at the row's own position is visible
    K3 = K.copy()
    K3[21] += 1.0
    o3, _ = causal_gqa_attention(q, pos, K3, V)
    assert not np.allclose(o3[5], o1[5]) and np.array_equal(o3[:5], o1[:5])
