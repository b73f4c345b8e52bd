"""Exact rational helpers for the oracle pins (pure Python, no oracle code).

These restate IEEE-754 rounding from its definition with ``fractions.Fraction``
so that the oracle's C arithmetic can be checked against something other than
itself.
"""
from __future__ import annotations

import math
import struct
from fractions import Fraction


def f32_bits(x: float) -> int:
    return struct.unpack("<I", struct.pack("<f", x))[0]


def bf16_value(h: int) -> Fraction:
    """Exact value of a BF16 bit pattern (finite)."""
    h = int(h)
    sign = -1 if (h >> 15) & 1 else 1
    ex = (h >> 7) & 0xFF
    fr = h & 0x7F
    assert ex != 0xFF, "not finite"
    if ex == 0:
        return sign * Fraction(fr, 1) * Fraction(2) ** (-126 - 7)
    return sign * Fraction(128 + fr) * Fraction(2) ** (ex - 127 - 7)


def floor_log2(a: Fraction) -> int:
    assert a > 0
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while a >= Fraction(2) ** (e + 1):
        e += 1
    while a < Fraction(2) ** e:
        e -= 1
    return e


def ceil_log2(a: Fraction) -> int:
    e = floor_log2(a)
    return e if a == Fraction(2) ** e else e + 1


def round_nearest_even(x: Fraction, p: int, emin: int, emax: int):
    """Round x to the binary format with p-bit significands, normal exponents
    emin..emax (subnormals below), ties to even.  Returns a Fraction, or
    +-inf (as float) on overflow."""
    if x == 0:
        return Fraction(0)
    s = -1 if x < 0 else 1
    a = abs(x)
    e = floor_log2(a)
    q = max(e, emin) - (p - 1)
    scaled = a / Fraction(2) ** q
    n = math.floor(scaled)
    rem = scaled - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = Fraction(n) * Fraction(2) ** q
    if r >= Fraction(2) ** (emax + 1):
        return s * math.inf
    return s * r


def to_f32(x: Fraction):
    return round_nearest_even(x, 24, -126, 127)


def to_bf16(x: Fraction):
    return round_nearest_even(x, 8, -126, 127)


def frac(x) -> Fraction:
    return Fraction(float(x))
