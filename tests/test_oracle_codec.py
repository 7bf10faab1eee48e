"""Pins for the oracle's binary16 codec (Section 3: IEEE 754 binary16).

Checked against (a) values fixed by the IEEE definition (golden file),
(b) the exhaustive set of 65,536 bit patterns, (c) numpy's own float16
conversion routines, and (d) the exact rational rounding in ``exact.py``.
"""

import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from exact import half_bits, half_value, to_half, to_half_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "binary16_values.txt")


def _golden():
    rows = []
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if not line:
            continue
        val, bits = line.split()[:2]
        if val.startswith("-0/"):
            v = -0.0
        else:
            v = float(Fraction(val))  # every golden value is exact in float64
            assert Fraction(v) == Fraction(val)
        rows.append((val, v, int(bits, 16)))
    return rows


@pytest.mark.parametrize("val,v,bits", _golden())
def test_known_values(val, v, bits):
    got = int(oracle.rne16(np.array([v])).view(np.uint16)[0])
    assert got == bits, f"{val}: got {got:#06x}, want {bits:#06x}"
    # the independent exact rounding agrees with the golden value
    if not val.startswith("-0/"):
        assert half_bits(to_half(Fraction(val))) == bits


def test_exhaustive_roundtrip():
    allbits = np.arange(65536, dtype=np.uint16)
    d = oracle.h2d(allbits)
    back = oracle.rne16(d).view(np.uint16)
    isnan = ((allbits & 0x7C00) == 0x7C00) & ((allbits & 0x3FF) != 0)
    assert np.array_equal(back[~isnan], allbits[~isnan])
    assert np.all(back[isnan] == 0x7E00)
    assert np.all(np.isnan(d[isnan]))


def test_decode_matches_numpy():
    allbits = np.arange(65536, dtype=np.uint16)
    d = oracle.h2d(allbits)
    ref = allbits.view(np.float16).astype(np.float64)
    ok = np.isnan(ref)
    assert np.array_equal(np.isnan(d), ok)
    assert np.array_equal(d[~ok], ref[~ok])
    assert np.array_equal(np.signbit(d[~ok]), np.signbit(ref[~ok]))


def test_decode_matches_exact_values():
    for b in list(range(0, 2048)) + list(range(0x3000, 0x3100)) + [0x7BFF, 0x7C00, 0xFC00, 0x8001]:
        v = half_value(b)
        got = oracle.h2d(np.array([b], np.uint16))[0]
        assert (Fraction(got) == v) if abs(v) != float("inf") else got == v


def _random_doubles(n, seed):
    rng = np.random.default_rng(seed)
    exps = rng.integers(-30, 18, size=n)
    mant = rng.random(n) + 1.0
    sign = np.where(rng.random(n) < 0.5, -1.0, 1.0)
    v = sign * np.ldexp(mant, exps)
    # add exact midpoints between neighbouring binary16 values (tie cases)
    h = rng.integers(0, 0x7BFF, size=n // 4).astype(np.uint16)
    lo = h.view(np.float16).astype(np.float64)
    hi = (h + 1).view(np.float16).astype(np.float64)
    mid = (lo + hi) / 2
    return np.concatenate([v, mid, -mid])


def test_random_doubles_match_numpy():
    v = _random_doubles(400_000, 1)
    got = oracle.rne16(v).view(np.uint16)
    with np.errstate(over="ignore"):
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)


def test_random_floats_match_numpy():
    v = _random_doubles(400_000, 2).astype(np.float32)
    got = oracle.rne16(v).view(np.uint16)
    with np.errstate(over="ignore"):
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)


def test_random_doubles_match_exact_rounding():
    v = _random_doubles(4000, 3)
    got = oracle.rne16(v).view(np.uint16)
    for x, g in zip(v, got):
        assert to_half_bits(Fraction(float(x))) == int(g), x


def test_nan_and_inf():
    got = oracle.rne16(np.array([np.nan, np.inf, -np.inf, 1e300, -1e300])).view(np.uint16)
    assert list(got) == [0x7E00, 0x7C00, 0xFC00, 0x7C00, 0xFC00]
