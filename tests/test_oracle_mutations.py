"""Planted mistakes in the oracle must be caught by its pins.

Each case swaps a deliberately wrong variant into the oracle (on the CPU) and
re-runs a pin from the other oracle test modules, expecting it to fail.
"""
import math

import numpy as np
import pytest

import test_oracle_attention as TA
import test_oracle_rope as TR
from oracle import attention as A
from oracle import rope as R


def _rope_variant(sign=1.0, interleaved=False, freq_scale=1.0):
    def f(x, positions, theta):
        x = np.asarray(x, dtype=np.float64)
        d = x.shape[-1]
        ang = np.asarray(positions, np.float64).reshape(-1, 1) * (
            R.inv_freq(d, theta) * freq_scale)[None, :]
        c, s = np.cos(ang)[:, None, :], sign * np.sin(ang)[:, None, :]
        if interleaved:
            a, b = x[..., 0::2], x[..., 1::2]
            y = np.empty_like(x)
            y[..., 0::2] = a * c - b * s
            y[..., 1::2] = b * c + a * s
            return y
        a, b = x[..., :d // 2], x[..., d // 2:]
        return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)
    return f


@pytest.mark.parametrize("kw", [dict(sign=-1.0), dict(interleaved=True),
                                dict(freq_scale=1.0001)])
def test_rope_mistakes_caught(monkeypatch, kw):
    monkeypatch.setattr(R, "rope_exact", _rope_variant(**kw))
    with pytest.raises(AssertionError):
        TR.test_matches_complex_exponential_form(10000.0)
        TR.test_d2_is_plane_rotation_by_p_radians()


def test_rope_fp32_with_fma_caught(monkeypatch):
    def fused(x, positions, theta):
        x64 = np.asarray(x, np.float32).astype(np.float64)
        c64, s64 = R.cos_sin_fp64(positions, x.shape[-1], theta)
        c = c64.astype(np.float32).astype(np.float64)[:, None, :]
        s = s64.astype(np.float32).astype(np.float64)[:, None, :]
        h = x.shape[-1] // 2
        a, b = x64[..., :h], x64[..., h:]
        lo = a * c - (b * s).astype(np.float32)
        hi = b * c + (a * s).astype(np.float32)
        return np.concatenate([lo, hi], -1).astype(np.float32)
    monkeypatch.setattr(R, "rope_fp32", fused)
    with pytest.raises(AssertionError):
        TR.test_fp32_is_no_fma_product_then_add()


def _attn_variant(strict=False, grouping="contiguous", scale_mul=1.0):
    def f(q, positions, K, V, scale=None, row_block=1024):
        q = np.asarray(q, np.float64)
        K = np.asarray(K, np.float64)
        V = np.asarray(V, np.float64)
        T, Hq, d = q.shape
        Hkv = K.shape[1]
        G = Hq // Hkv
        sc = (1.0 / math.sqrt(d) if scale is None else scale) * scale_mul
        out = np.zeros((T, Hq, d))
        lse = np.zeros((T, Hq))
        for t in range(T):
            p = int(positions[t])
            n = p if strict else p + 1
            n = max(n, 1)
            for h in range(Hq):
                g = h // G if grouping == "contiguous" else h % Hkv
                s = sc * (K[:n, g] @ q[t, h])
                e = np.exp(s - s.max())
                out[t, h] = e @ V[:n, g] / e.sum()
                lse[t, h] = s.max() + np.log(e.sum())
        return out, lse
    return f


@pytest.mark.parametrize("kw,pin", [
    (dict(strict=True), "test_matches_brute_force_loops"),
    (dict(grouping="modulo"), "test_matches_torch_sdpa_float64"),
    (dict(scale_mul=1.01), "test_matches_brute_force_loops"),
])
def test_attention_mistakes_caught(monkeypatch, kw, pin):
    monkeypatch.setattr(TA, "causal_gqa_attention", _attn_variant(**kw))
    fn = getattr(TA, pin)
    with pytest.raises(AssertionError):
        if pin == "test_matches_torch_sdpa_float64":
            fn(8, 2)
        else:
            fn()
