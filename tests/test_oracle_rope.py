"""Pins for oracle.rope (RoPE of Section 2.2: rotate q and k, not v)."""
import math

import numpy as np
import pytest

from oracle import rope as R

THETAS = [10000.0, 500000.0]


def test_inv_freq_closed_form():
    # theta^(-2i/d) == exp(-(2i/d) ln theta), evaluated through exp/log
    for theta in THETAS:
        for d in (2, 64, 128):
            i = np.arange(d // 2)
            ref = np.exp(-(2.0 * i / d) * np.log(theta))
            assert np.allclose(R.inv_freq(d, theta), ref, rtol=1e-14, atol=0)
            assert R.inv_freq(d, theta)[0] == 1.0


def test_d2_is_plane_rotation_by_p_radians():
    x = np.array([[[0.3, -1.7]]])
    for p in (0, 1, 5, 1000, 33000):
        y = R.rope_exact(x, [p], 10000.0)[0, 0]
        c, s = math.cos(p), math.sin(p)
        assert np.allclose(y, [0.3 * c + 1.7 * s, -1.7 * c + 0.3 * s], rtol=0, atol=1e-12)


@pytest.mark.parametrize("theta", THETAS)
def test_matches_complex_exponential_form(theta):
    rng = np.random.default_rng(0)
    x = rng.standard_normal((50, 3, 128))
    pos = rng.integers(0, 40000, 50)
    assert np.allclose(R.rope_exact(x, pos, theta), R.rope_complex(x, pos, theta),
                       rtol=0, atol=1e-10)


def test_identity_at_zero_and_norm_preserved():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((8, 2, 64))
    assert np.array_equal(R.rope_exact(x, np.zeros(8, int), 1e4), x)
    y = R.rope_exact(x, np.arange(8) * 977, 1e4)
    a, b = x[..., :32], x[..., 32:]
    ya, yb = y[..., :32], y[..., 32:]
    assert np.allclose(a**2 + b**2, ya**2 + yb**2, rtol=1e-13)


@pytest.mark.parametrize("theta", THETAS)
def test_rotations_compose_additively(theta):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((20, 4, 128))
    a = rng.integers(0, 20000, 20)
    b = rng.integers(0, 20000, 20)
    two = R.rope_exact(R.rope_exact(x, a, theta), b, theta)
    one = R.rope_exact(x, a + b, theta)
    assert np.allclose(two, one, rtol=0, atol=1e-9)


@pytest.mark.parametrize("theta", THETAS)
def test_scores_depend_only_on_relative_offset(theta):
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 1, 128))
    k = rng.standard_normal((1, 1, 128))
    base = None
    for p1 in (100, 5000, 31000):
        p2 = p1 - 77
        s = float(np.sum(R.rope_exact(q, [p1], theta) * R.rope_exact(k, [p2], theta)))
        base = s if base is None else base
        assert abs(s - base) < 1e-9 * max(1.0, abs(base))


def test_v_untouched_is_a_property_of_the_path_not_rope():
    # RoPE acts on pairs (i, i+d/2); with d/2 pairs every dimension is rotated
    x = np.eye(8).reshape(8, 1, 8)
    y = R.rope_exact(x, np.full(8, 3), 1e4)
    assert not np.allclose(y, x)


@pytest.mark.parametrize("theta", THETAS)
def test_rerotation_of_cached_key_matches_direct_encoding(theta):
    """A key cached before RoPE and rotated at its new offset equals the key
    encoded directly at that offset (fp32 evaluation: within 2 ulp of the
    fp64 definition, and identical between the two routes)."""
    rng = np.random.default_rng(4)
    k = rng.standard_normal((300, 8, 128)).astype(np.float32)
    new_pos = rng.integers(0, 33000, 300)
    fp32 = R.rope_fp32(k, new_pos, theta)
    exact = R.rope_exact(k, new_pos, theta)
    # fp32 evaluation error: 2 roundings of products + 1 of the sum, plus
    # table rounding -> bounded by a few ulp of the operands' magnitude
    ulp = np.spacing(np.abs(k).max(axis=-1, keepdims=True).astype(np.float32))
    assert np.all(np.abs(fp32 - exact) <= 4 * ulp)
    # a key rotated by its cached offset 0 first (identity) then re-rotated
    # to p matches direct rotation at p bit for bit
    at0 = R.rope_fp32(k, np.zeros(300, int), theta)
    assert np.array_equal(at0, k)
    assert np.array_equal(R.rope_fp32(at0, new_pos, theta), fp32)


def test_fp32_is_no_fma_product_then_add():
    # scalar fp32 evaluation pair by pair: each product rounded, then the sum
    rng = np.random.default_rng(9)
    n, d = 1000, 2
    x = rng.standard_normal((n, 1, d)).astype(np.float32)
    pos = rng.integers(0, 40000, n)
    got = R.rope_fp32(x, pos, 10000.0)[:, 0]
    for t in range(n):
        c, s = np.float32(math.cos(pos[t])), np.float32(math.sin(pos[t]))
        a, b = x[t, 0, 0], x[t, 0, 1]
        lo = np.float32(np.float32(a * c) - np.float32(b * s))
        hi = np.float32(np.float32(b * c) + np.float32(a * s))
        assert got[t, 0] == lo and got[t, 1] == hi, t
