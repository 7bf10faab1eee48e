"""Exact rational arithmetic for pinning the oracle.

An independent, integer-only implementation of IEEE 754 round-to-nearest,
ties-to-even for binary16 and binary32, used to check the oracle's own codec
and its declared float32 sequences.  Shares nothing with the oracle.
"""

from __future__ import annotations

from fractions import Fraction

INF = float("inf")


def _floor_log2(q: Fraction) -> int:
    a, b = q.numerator, q.denominator
    e = a.bit_length() - b.bit_length()
    # ensure 2^e <= a/b < 2^(e+1)
    if e >= 0:
        if a < (b << e):
            e -= 1
    else:
        if (a << -e) < b:
            e -= 1
    return e


def round_binary(q: Fraction, p: int, emin: int, emax: int):
    """Round the rational q to a binary format with p significand bits.

    Returns a Fraction, or +-INF on overflow.  Ties go to the even
    significand; values below 2^emin keep the fixed quantum 2^(emin-p+1)
    (gradual underflow)."""
    if q == 0:
        return Fraction(0)
    sign = -1 if q < 0 else 1
    a = abs(q)
    e = max(_floor_log2(a), emin)
    quantum = Fraction(1, 1) * (Fraction(2) ** (e - p + 1))
    units = a / quantum
    n, rem = divmod(units.numerator, units.denominator)
    frac = Fraction(rem, units.denominator)
    if frac > Fraction(1, 2) or (frac == Fraction(1, 2) and n % 2 == 1):
        n += 1
    r = n * quantum
    if r >= Fraction(2) ** (emax + 1):
        return sign * INF
    return sign * r


def to_half(q: Fraction):
    return round_binary(q, 11, -14, 15)


def to_single(q: Fraction):
    return round_binary(q, 24, -126, 127)


def half_bits(v) -> int:
    """binary16 encoding of an exactly representable value (Fraction or +-inf)."""
    if v == INF:
        return 0x7C00
    if v == -INF:
        return 0xFC00
    v = Fraction(v)
    sign = 0x8000 if v < 0 else 0
    a = abs(v)
    if a == 0:
        return sign
    if a < Fraction(1, 2 ** 14):
        units = a * 2 ** 24
        assert units.denominator == 1
        return sign | int(units)
    e = _floor_log2(a)
    sig = a / Fraction(2) ** (e - 10)
    assert sig.denominator == 1 and 1024 <= sig < 2048
    return sign | ((e + 15) << 10) | (int(sig) - 1024)


def to_half_bits(q: Fraction) -> int:
    """binary16 bits of q rounded to nearest even; a negative q that rounds
    to zero gives -0 (0x8000), as IEEE rounding keeps the sign."""
    b = half_bits(to_half(q))
    if q < 0 and b == 0:
        return 0x8000
    return b


def half_value(bits: int):
    """Exact value of a (non-NaN) binary16 bit pattern."""
    sign = -1 if bits & 0x8000 else 1
    e = (bits >> 10) & 31
    f = bits & 1023
    if e == 31:
        assert f == 0, "NaN has no exact value"
        return sign * INF
    if e == 0:
        return sign * Fraction(f, 2 ** 24)
    return sign * Fraction(1024 + f) * Fraction(2) ** (e - 25)
