"""Storage-format rounding for the oracle (bf16, OCP e4m3fn).

The paper stores 16-bit KV states (Section 2.4); the exact 16-bit format is
not stated.  bf16 is used here, rounded to nearest-even from fp32.  The fp8
pool variant uses OCP e4m3fn (1 sign, 4 exponent bits with bias 7, 3 mantissa
bits, no infinities, max finite 448), rounded to nearest-even and saturating
to +-448 -- a reading, since the paper has no fp8 path.

Both encoders are written from the format definitions by integer arithmetic
on the IEEE fp32 bit pattern.  Pins: tests/test_oracle_numerics.py compares
them with torch's CPU conversions (a library routine) on random and edge
values.
"""
from __future__ import annotations

import numpy as np


# ----------------------------------------------------------------- bfloat16
def f32_to_bf16_bits(x) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return uint16 bits.

    bf16 keeps the top 16 bits of the fp32 pattern.  Rounding adds half of
    the dropped range (0x7FFF) plus the lowest kept bit (ties to even) before
    truncation; a carry into the exponent is the correct overflow to the next
    binade or to infinity.  NaN is kept quiet.
    """
    b = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    is_nan = (b & 0x7F800000) == 0x7F800000
    is_nan &= (b & 0x007FFFFF) != 0
    lsb = (b >> 16) & 1
    r = ((b + 0x7FFF + lsb) >> 16) & 0xFFFF
    r = np.where(is_nan, (b >> 16) | 0x0040, r)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def round_bf16(x) -> np.ndarray:
    """fp32 -> bf16 -> fp32 (values as float32)."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


# ---------------------------------------------------------- OCP e4m3 (fn)
E4M3_MAX = 448.0


def e4m3_decode(codes) -> np.ndarray:
    """uint8 e4m3fn codes -> float32 values (0x7F / 0xFF are NaN)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    normal = np.ldexp(1.0 + m / 8.0, e - 7)
    sub = np.ldexp(m / 8.0, -6)
    v = sign * np.where(e == 0, sub, normal)
    v = np.where((c & 0x7F) == 0x7F, np.nan, v)
    return v.astype(np.float32)


def e4m3_encode(x) -> np.ndarray:
    """float32 -> e4m3fn code, nearest-even, saturating to +-448.

    The representable magnitudes are k * 2^(e-3) for 8 <= k < 16 in binade
    e >= -6, and k * 2^-9 for 0 <= k < 8 (subnormals).  Rounding is done on
    the integer k at the binade's quantum, which is exact in fp64.
    """
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    nan = np.isnan(x)
    sign = np.signbit(x)
    a = np.minimum(np.abs(np.where(nan, 0.0, x)), E4M3_MAX)
    # binade exponent of a (a >= 2^-6 normal), clamped to the subnormal binade
    e = np.floor(np.log2(np.where(a > 0, a, 1.0))).astype(np.int64)
    # guard log2 rounding at exact powers of two
    e = np.where(np.ldexp(1.0, e) > a, e - 1, e)
    e = np.where(np.ldexp(1.0, e + 1) <= a, e + 1, e)
    e = np.maximum(e, -6)
    quantum = np.ldexp(1.0, e - 3)
    k = a / quantum                          # exact: power-of-two divide
    kr = np.round(k)                         # numpy rounds half to even
    # rounding up to 16 quanta moves to the next binade (k = 8 there)
    bump = kr >= 16
    e = np.where(bump, e + 1, e)
    kr = np.where(bump, 8, kr).astype(np.int64)
    is_sub = (e == -6) & (kr < 8)
    exp_field = np.where(is_sub, 0, e + 7)
    man = np.where(is_sub, kr, kr - 8)
    code = (exp_field << 3) | man
    code = np.where(a == 0, 0, code)
    code = code | np.where(sign, 0x80, 0)
    code = np.where(nan, 0x7F, code)
    return code.astype(np.uint8)


def e4m3_page_scale(amax) -> np.ndarray:
    """Per-page power-of-two scale: the smallest 2^k with amax / 2^k <= 448.

    scale = 2^ceil(log2(amax / 448)); 1.0 when amax == 0.  Dividing by a
    power of two is exact, so quantization error comes only from rounding to
    e4m3.  (A reading: the paper has no fp8 path.)
    """
    amax = np.asarray(amax, dtype=np.float64)
    out = np.ones_like(amax)
    nz = amax > 0
    k = np.ceil(np.log2(amax[nz] / E4M3_MAX)).astype(np.int64)
    # guard the ceil against log2 rounding: enforce amax / 2^k <= 448 minimal
    s = np.ldexp(1.0, k)
    k = np.where(amax[nz] / s > E4M3_MAX, k + 1, k)
    s = np.ldexp(1.0, k)
    k = np.where(amax[nz] / np.ldexp(1.0, k - 1) <= E4M3_MAX, k - 1, k)
    out[nz] = np.ldexp(1.0, k)
    return out.astype(np.float32)


# ---------------------------------------------------------------- float16
def round_f16(x) -> np.ndarray:
    """fp32 -> IEEE binary16 (numpy's nearest-even conversion) -> fp32."""
    return np.asarray(x, dtype=np.float32).astype(np.float16).astype(np.float32)
