"""Pins for oracle.numerics: storage-format rounding vs torch's CPU casts."""
import numpy as np
import pytest
import torch

from oracle import numerics as N


def _edge_f32():
    vals = [0.0, -0.0, 1.0, -1.0, 1 + 2**-8, 1 + 3 * 2**-8, 1 + 2**-9, 65504.0,
            3.3895313892515355e38, 3.4e38, 1e-40, -1e-40, 2**-126, 2**-133,
            float("inf"), float("-inf")]
    return np.array(vals, dtype=np.float32)


def test_bf16_matches_torch_edges():
    x = _edge_f32()
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(N.f32_to_bf16_bits(x), ref)


def test_bf16_matches_torch_random_bits():
    rng = np.random.default_rng(5)
    bits = rng.integers(0, 2**32, size=200000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[~np.isnan(x)]
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(N.f32_to_bf16_bits(x), ref)


def test_bf16_ties_to_even():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to the even mantissa (1.0)
    assert N.round_bf16(np.float32(1 + 2**-8)) == np.float32(1.0)
    # 1 + 3*2^-8 is halfway between 1+2^-7 and 1+2^-6: rounds up to even 1+2^-6
    assert N.round_bf16(np.float32(1 + 3 * 2**-8)) == np.float32(1 + 2**-6)


def test_bf16_nan_stays_nan():
    assert np.isnan(N.round_bf16(np.float32("nan")))


def test_e4m3_decode_all_codes_match_torch():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float32).numpy()
    got = N.e4m3_decode(codes)
    assert np.array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(got[ok], ref[ok])


def test_e4m3_encode_matches_torch_in_range():
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.standard_normal(100000) * s for s in (1e-3, 0.1, 1, 30, 200)])
    x = np.clip(x, -448, 448).astype(np.float32)
    # every midpoint between consecutive codes, both signs (ties to even)
    vals = np.unique(N.e4m3_decode(np.arange(0, 0x7F, dtype=np.uint8)))
    mids = ((vals[1:].astype(np.float64) + vals[:-1]) / 2).astype(np.float32)
    x = np.concatenate([x, mids, -mids, vals, -vals])
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = N.e4m3_encode(x)
    # +-0 may differ in sign handling only for -0.0; compare values
    assert np.array_equal(N.e4m3_decode(got), N.e4m3_decode(ref))


def test_e4m3_saturates():
    x = np.array([449.0, 1000.0, -1e9, 464.0, 480.0], dtype=np.float32)
    got = N.e4m3_decode(N.e4m3_encode(x))
    assert np.array_equal(got, np.array([448, 448, -448, 448, 448], dtype=np.float32))


@pytest.mark.parametrize("amax", [0.0, 1e-8, 0.3, 1.0, 447.9, 448.0, 448.1, 896.0, 1e6])
def test_e4m3_page_scale_is_minimal_power_of_two(amax):
    s = float(N.e4m3_page_scale(np.array([amax]))[0])
    if amax == 0:
        assert s == 1.0
        return
    m, e = np.frexp(s)
    assert m == 0.5                       # a power of two
    assert amax / s <= 448.0
    assert amax / (s / 2) > 448.0         # the next smaller power would overflow


def test_round_f16_is_ieee():
    x = np.array([1 + 2**-11, 1 + 3 * 2**-11, 65504, 65520, 6e-8], dtype=np.float32)
    ref = torch.from_numpy(x).to(torch.float16).to(torch.float32).numpy()
    assert np.array_equal(N.round_f16(x), ref)
