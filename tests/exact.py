"""Exact-arithmetic references used to pin the oracle's fp8 cast.

Everything here uses Python's ``fractions.Fraction``: values are exact
rationals, binary32 rounding is done by hand from its definition (nearest
representable, ties to an even significand) and the E4M3 encoding is a
search for the nearest of all finite codes by exact distance.  None of it
uses a floating-point division, a bit trick or the oracle's code.
"""
from __future__ import annotations

import bisect
import math
import struct
from fractions import Fraction


def f32_bits(x: float) -> int:
    return struct.unpack("<I", struct.pack("<f", x))[0]


def bits_f32(u: int) -> float:
    return struct.unpack("<f", struct.pack("<I", u & 0xFFFFFFFF))[0]


def bf16_to_float(bits: int) -> float:
    return bits_f32((bits & 0xFFFF) << 16)


def e4m3_value(code: int):
    """Value of an E4M3 code from the format definition (None for NaN)."""
    s = -1 if code & 0x80 else 1
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return None
    if e == 0:
        return s * Fraction(m, 8) * Fraction(1, 2 ** 6)
    return s * (1 + Fraction(m, 8)) * Fraction(2) ** (e - 7)


# Finite non-negative magnitudes with their codes, sorted by value.
_POS = sorted((e4m3_value(c), c) for c in range(0x00, 0x7F))
_POS_VALS = [v for v, _ in _POS]
MAX_FINITE = _POS_VALS[-1]


def nearest_e4m3(v, negative: bool) -> int:
    """Code of the finite E4M3 value nearest to the exact rational |v| (>= 0),
    ties to the code with an even mantissa, saturating beyond 448."""
    a = abs(Fraction(v))
    sign = 0x80 if negative else 0x00
    if a >= MAX_FINITE:
        return sign | 0x7E
    k = bisect.bisect_right(_POS_VALS, a) - 1  # _POS_VALS[k] <= a
    cands = [_POS[k]]
    if k + 1 < len(_POS):
        cands.append(_POS[k + 1])
    best = min(abs(a - val) for val, _ in cands)
    winners = [c for val, c in cands if abs(a - val) == best]
    if len(winners) > 1:
        winners = [c for c in winners if (c & 1) == 0]
    return sign | winners[0]


def encode_float(x: float) -> int:
    """E4M3 code of a (binary32) float, with NaN -> 0x7F and Inf saturating."""
    if math.isnan(x):
        return 0x7F
    neg = math.copysign(1.0, x) < 0
    if math.isinf(x):
        return (0x80 if neg else 0) | 0x7E
    return nearest_e4m3(Fraction(x), neg)


def rn_f32(v: Fraction, negative_zero: bool = False) -> float:
    """Round an exact rational to the nearest binary32 value, ties to even,
    with gradual underflow and overflow to infinity."""
    if v == 0:
        return -0.0 if negative_zero else 0.0
    neg = v < 0
    a = -v if neg else v
    e = a.numerator.bit_length() - a.denominator.bit_length()
    two = Fraction(2)
    while two ** e > a:
        e -= 1
    while two ** (e + 1) <= a:
        e += 1
    e = max(e, -126)                   # below 2^-126 the quantum stays 2^-149
    quantum = two ** (e - 23)
    m = a / quantum
    n = m.numerator // m.denominator
    rem = m - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    val = n * quantum
    if val >= two ** 128:
        out = math.inf
    else:
        out = float(val)               # exact: val is a binary32 value
    return -out if neg else out


def quotient_code(x: float, s: float) -> int:
    """E4M3 code of RN_f32(x / s) for finite x and finite non-zero s."""
    neg = (math.copysign(1.0, x) < 0) != (s < 0)
    q = rn_f32(Fraction(x) / Fraction(s), negative_zero=neg)
    return encode_float(q)


def rn_bf16_of_f32(x: float) -> int:
    """bf16 bit pattern of a binary32 value rounded to 8 significant bits
    (nearest, ties to even), computed on the exact value; NaN -> 0x7FC0."""
    if math.isnan(x):
        return 0x7FC0
    sign = 0x8000 if math.copysign(1.0, x) < 0 else 0
    if math.isinf(x):
        return sign | 0x7F80
    a = Fraction(abs(x))
    if a == 0:
        return sign
    two = Fraction(2)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while two ** e > a:
        e -= 1
    while two ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    quantum = two ** (e - 7)                  # 8 significant bits
    m = a / quantum
    n = m.numerator // m.denominator
    rem = m - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    val = n * quantum
    if val >= two ** 128:
        return sign | 0x7F80
    return sign | (f32_bits(float(val)) >> 16)
