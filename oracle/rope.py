"""Rotary position encoding (RoPE) for the oracle.

The paper targets RoPE models, which rotate queries and keys but not values,
and caches keys before RoPE so that they can be rotated for a unit's new
offset (Section 2.2; Section 5.1 "Per-unit plan": the reusable form is the
keys before RoPE together with the values).  The variant is not stated; the
reading here is the textbook rotation used by Llama-family models:

* pair i (0 <= i < d/2) couples dimensions i and i + d/2 ("half-split");
* its frequency is theta^(-2i/d), its angle at position p is p * theta^(-2i/d);
* (x_i, x_{i+d/2}) -> (x_i cos - x_{i+d/2} sin, x_{i+d/2} cos + x_i sin),
  i.e. multiplication of x_i + 1j x_{i+d/2} by exp(1j * angle).

Two evaluations are provided:
* rope_exact: fp64 throughout (the definition);
* rope_fp32: the fp64 cos/sin rounded to fp32, then fp32 products and one
  fp32 add/subtract each, no fused multiply-add.  This is the reference a
  GPU kernel built on an fp32 cos/sin table can match bit for bit.

Pins (tests/test_oracle_rope.py): complex-exponential form at d = 2 and at
full width, identity at p = 0, norm preservation, R(a)R(b) = R(a+b),
dependence of <R(p1)q, R(p2)k> on p1 - p2 only, and re-rotation of a key
cached before RoPE equals direct encoding at the new position.
"""
from __future__ import annotations

import math

import numpy as np

_TABLES: dict[tuple[int, float], tuple[np.ndarray, np.ndarray]] = {}


def inv_freq(head_dim: int, theta: float) -> np.ndarray:
    """fp64 frequencies theta^(-2i/d), i = 0 .. d/2-1 (libm pow)."""
    if head_dim % 2:
        raise ValueError("head_dim must be even")
    return np.array([math.pow(theta, -2.0 * i / head_dim)
                     for i in range(head_dim // 2)], dtype=np.float64)


def angles(positions, head_dim: int, theta: float) -> np.ndarray:
    """fp64 angles [n][d/2] = p * theta^(-2i/d)."""
    p = np.asarray(positions, dtype=np.float64).reshape(-1, 1)
    return p * inv_freq(head_dim, theta).reshape(1, -1)


def cos_sin_fp64(positions, head_dim: int, theta: float):
    """fp64 cos and sin of the angles, [n][d/2] each (libm cos / sin).

    Values for positions 0 .. max are cached per (d, theta).
    """
    positions = np.asarray(positions, dtype=np.int64)
    need = int(positions.max()) + 1 if positions.size else 0
    key = (int(head_dim), float(theta))
    c, s = _TABLES.get(key, (np.zeros((0, head_dim // 2)),) * 2)
    if c.shape[0] < need:
        n0 = c.shape[0]
        ang = angles(np.arange(n0, need), head_dim, theta)
        flat = ang.ravel()
        cn = np.fromiter((math.cos(a) for a in flat), np.float64, flat.size)
        sn = np.fromiter((math.sin(a) for a in flat), np.float64, flat.size)
        c = np.concatenate([c, cn.reshape(ang.shape)])
        s = np.concatenate([s, sn.reshape(ang.shape)])
        _TABLES[key] = (c, s)
    return c[positions], s[positions]


def _split(x):
    h = x.shape[-1] // 2
    return x[..., :h], x[..., h:]


def rope_exact(x, positions, theta: float) -> np.ndarray:
    """fp64 RoPE of x [n][H][d] at positions [n]."""
    x = np.asarray(x, dtype=np.float64)
    c, s = cos_sin_fp64(positions, x.shape[-1], theta)
    c, s = c[:, None, :], s[:, None, :]
    a, b = _split(x)
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def rope_fp32(x, positions, theta: float) -> np.ndarray:
    """RoPE in fp32 arithmetic from an fp32 cos/sin table, no FMA.

    Every product is rounded to fp32, then the two products are added or
    subtracted with one more fp32 rounding.
    """
    x = np.asarray(x, dtype=np.float32)
    c64, s64 = cos_sin_fp64(positions, x.shape[-1], theta)
    c = c64.astype(np.float32)[:, None, :]
    s = s64.astype(np.float32)[:, None, :]
    a, b = _split(x)
    lo = (a * c) - (b * s)
    hi = (b * c) + (a * s)
    return np.concatenate([lo, hi], axis=-1).astype(np.float32)


def rope_complex(x, positions, theta: float) -> np.ndarray:
    """fp64 RoPE written as complex multiplication (used to pin rope_exact)."""
    x = np.asarray(x, dtype=np.float64)
    a, b = _split(x)
    z = (a + 1j * b) * np.exp(1j * angles(positions, x.shape[-1], theta))[:, None, :]
    return np.concatenate([z.real, z.imag], axis=-1)
