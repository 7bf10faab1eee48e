"""Pins for the oracle's strict binary16 arithmetic (all operations in FP16,
the literal reading of Section 5.2), used to measure what the float32
accumulators of the default path buy.

- fma16: exact rational evaluation (tests/exact.py) of round(a*b + c) on
  random and constructed binary16 triples, including subnormals, overflow
  and halfway cases.
- SGD with binary16 arithmetic: exact rational evaluation of the three
  fused multiply-adds with binary16 scalars; one hand-derived example where
  the extra rounding of d changes the momentum by one ulp.
- Convolutions with a binary16 accumulator rounded once per 16 terms:
  (a) with at most 16 terms there is one rounding, so the result equals the
      (separately pinned) single rounding of the exact sum;
  (b) on small-integer data every partial sum is a binary16 integer, so the
      result is exact;
  (c) an independent brute force on tiny shapes -- the reduction written
      out as an explicit im2col row for the forward and the weight gradient,
      and for the data gradient as the list of forward contributions that
      reach the position, sorted by the declared key -- accumulated in exact
      rationals with one binary16 rounding per block of 16.
"""

from fractions import Fraction

import numpy as np
import pytest

import oracle
from exact import half_value, to_half_bits
from paper_1911_07384_amd import synth


def _rand_bits(rng, n, lo_exp=-24, hi_exp=15):
    """Random finite binary16 patterns with log-uniform magnitudes."""
    e = rng.integers(lo_exp, hi_exp + 1, n)
    v = rng.uniform(1, 2, n) * (2.0 ** e) * rng.choice([-1, 1], n)
    b = np.clip(v, -65504, 65504).astype(np.float16).view(np.uint16)
    return b


def _fma_exact(a, b, c):
    q = half_value(int(a)) * half_value(int(b)) + half_value(int(c))
    return q


def _check_fma(a, b, c):
    got = oracle.fma16(a.view(np.float16), b.view(np.float16), c.view(np.float16)).view(np.uint16)
    for i in range(a.size):
        q = _fma_exact(a[i], b[i], c[i])
        if q == 0:
            # exact zero: +0 unless both the product and c are -0 (IEEE sum rules)
            prod_neg = (int(a[i]) ^ int(b[i])) & 0x8000
            both_neg_zero = prod_neg and (int(c[i]) & 0x8000) and half_value(int(c[i])) == 0
            assert int(got[i]) == (0x8000 if both_neg_zero else 0), (a[i], b[i], c[i], got[i])
        else:
            assert int(got[i]) == to_half_bits(q), (hex(a[i]), hex(b[i]), hex(c[i]), hex(got[i]))


def test_fma16_random_matches_exact():
    rng = np.random.default_rng(5)
    n = 20000
    _check_fma(_rand_bits(rng, n, -12, 8), _rand_bits(rng, n, -12, 8), _rand_bits(rng, n, -24, 15))


def test_fma16_subnormal_and_overflow_matches_exact():
    rng = np.random.default_rng(6)
    n = 5000
    # products in the subnormal range, sums near the overflow threshold
    _check_fma(_rand_bits(rng, n, -24, -8), _rand_bits(rng, n, -10, 0), _rand_bits(rng, n, -24, -14))
    _check_fma(_rand_bits(rng, n, 6, 8), _rand_bits(rng, n, 6, 8), _rand_bits(rng, n, 14, 15))


def test_fma16_halfway_cases():
    one = np.float16(1.0).view(np.uint16)
    # 1 + 2^-11 is halfway between 1 and 1 + 2^-10
    a = np.array([np.float16(2.0 ** -11).view(np.uint16)] * 3, np.uint16)
    b = np.array([np.float16(1.0), np.float16(1.0 + 2.0 ** -10), np.float16(1.0 - 2.0 ** -11)],
                 np.float16).view(np.uint16)
    c = np.array([one] * 3, np.uint16)
    got = oracle.fma16(a.view(np.float16), b.view(np.float16), c.view(np.float16)).view(np.uint16)
    # exact tie -> even (1.0); just above -> up; just below -> down
    assert [int(v) for v in got] == [0x3C00, 0x3C01, 0x3C00]
    _check_fma(a, b, c)


def _sgd_exact(w, g, m, lr, mom, wd):
    f32 = lambda v: Fraction(float(np.float32(v)))
    lam = half_value(to_half_bits(f32(wd)))
    mu = half_value(to_half_bits(f32(mom)))
    nlr = half_value(to_half_bits(-f32(lr)))
    d = to_half_bits(lam * half_value(w) + half_value(g))
    m1 = to_half_bits(mu * half_value(m) + half_value(d))
    w1 = to_half_bits(nlr * half_value(m1) + half_value(w))
    return w1, m1


def test_sgd_f16_matches_exact():
    rng = np.random.default_rng(7)
    n = 3000
    w = (rng.standard_normal(n) * 0.05).astype(np.float16)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float16)
    m = (rng.standard_normal(n) * 1e-2).astype(np.float16)
    for lr, mom, wd in [(0.1, 0.9, 1e-4), (2.0 ** -14, 0.9, 1e-4), (0.1, 0.9, 0.0)]:
        w1, m1 = oracle.sgd_f16(w, g, m, lr, mom, wd)
        for i in range(n):
            ew, em = _sgd_exact(int(w.view(np.uint16)[i]), int(g.view(np.uint16)[i]),
                                int(m.view(np.uint16)[i]), lr, mom, wd)
            assert int(w1.view(np.uint16)[i]) == ew and int(m1.view(np.uint16)[i]) == em, (i, lr)


def test_sgd_f16_worked_example():
    # w = 1, g = 2^-12, m = 0, lr = 0.1, momentum 0.9, weight decay 1e-4.
    # binary16 weight decay: 1e-4 (float32) -> 1678 * 2^-24.  d = 2^-12 + 1678 * 2^-24
    # = (4096 + 1678) * 2^-24 = 5774 * 2^-24; the binary16 quantum in
    # [2^-12, 2^-11) is 2^-22, so d = round(1443.5) * 2^-22 -> 1444 * 2^-22
    # (a tie, to even).  m' = 0.9 * 0 + d = 1444 * 2^-22 = 0x0DA4.
    # The float32 sequence keeps d unrounded and rounds 1443.5 (plus the
    # float32 error of 1e-4) once at m': 0x0DA3 -- one ulp apart.
    w = np.array([1.0], np.float16)
    g = np.array([2.0 ** -12], np.float16)
    m = np.zeros(1, np.float16)
    _, m_strict = oracle.sgd_f16(w, g, m, 0.1, 0.9, 1e-4)
    _, m_f32 = oracle.sgd_f32(w, g, m, 0.1, 0.9, 1e-4)
    assert int(m_strict.view(np.uint16)[0]) == 0x0DA4
    assert int(m_f32.view(np.uint16)[0]) == 0x0DA3


# ---- convolutions ---------------------------------------------------------

def _inputs(shp, seed, grid=None, scale=1.0):
    n, c, h, w, k, r, s = (int(v) for v in shp[:7])
    p, q = oracle.conv_out_dims(shp)
    x = synth.normal_f16((n, h, w, c), 1.0, seed, 1)
    wt = synth.normal_f16((k, r, s, c), scale * synth.he_std(c * r * s), seed, 2)
    dy = synth.normal_f16((n, p, q, k), 1.0, seed, 3)
    if grid is not None:
        rng = np.random.default_rng(seed)
        x = rng.integers(-grid, grid + 1, x.shape).astype(np.float16)
        wt = rng.integers(-grid, grid + 1, wt.shape).astype(np.float16)
        dy = rng.integers(-grid, grid + 1, dy.shape).astype(np.float16)
    return x, wt, dy


@pytest.mark.parametrize("c,k", [(8, 4), (16, 16), (3, 5)])
def test_single_block_equals_one_rounding(c, k):
    # 1x1: the forward reduction has Cp <= 16 terms, the data gradient Kp <= 16,
    # the weight gradient N*P*Q <= 16 pixels
    shp = oracle.conv_shape(1, c, 4, 4, k, 1, 1)
    x, w, dy = _inputs(shp, 11)
    assert np.array_equal(oracle.conv_fwd_f16acc(shp, x, w).view(np.uint16),
                          oracle.conv_fwd(shp, x, w)[1].view(np.uint16))
    assert np.array_equal(oracle.conv_dgrad_f16acc(shp, dy, w).view(np.uint16),
                          oracle.conv_dgrad(shp, dy, w)[1].view(np.uint16))
    assert np.array_equal(oracle.conv_wgrad_f16acc(shp, x, dy).view(np.uint16),
                          oracle.conv_wgrad(shp, x, dy)[1].view(np.uint16))


@pytest.mark.parametrize("shape", [(2, 24, 7, 6, 10, 3, 3, 1, 1), (2, 16, 9, 9, 8, 3, 3, 2, 1),
                                   (1, 8, 5, 5, 12, 1, 1, 2, 0)])
def test_integer_grid_is_exact(shape):
    n, c, h, w, k, r, s, st, pad = shape
    shp = oracle.conv_shape(n, c, h, w, k, r, s, st, pad)
    x, wt, dy = _inputs(shp, 12, grid=2)
    for strict, (ref64, _) in [(oracle.conv_fwd_f16acc(shp, x, wt), oracle.conv_fwd(shp, x, wt)),
                               (oracle.conv_dgrad_f16acc(shp, dy, wt), oracle.conv_dgrad(shp, dy, wt)),
                               (oracle.conv_wgrad_f16acc(shp, x, dy), oracle.conv_wgrad(shp, x, dy))]:
        assert np.abs(ref64).max() < 2048  # every partial sum is a binary16 integer
        assert np.array_equal(strict.astype(np.float64), ref64)


def _blocks16(terms):
    """Binary16 accumulator updated once per block of 16 exact terms."""
    acc = Fraction(0)
    for i in range(0, len(terms), 16):
        acc = half_value(to_half_bits(acc + sum(terms[i:i + 16], Fraction(0))))
    return to_half_bits(acc)


def _hv(a):
    return [half_value(int(b)) for b in np.ascontiguousarray(a).view(np.uint16).reshape(-1)]


@pytest.mark.parametrize("shape", [(1, 3, 5, 5, 4, 3, 3, 1, 1), (2, 8, 6, 5, 3, 3, 3, 2, 1),
                                   (1, 5, 7, 7, 2, 3, 3, 2, 0), (1, 16, 4, 4, 8, 1, 1, 2, 0)])
def test_brute_force_block_order(shape):
    n, c, h, w, k, r, s, st, pad = shape
    shp = oracle.conv_shape(n, c, h, w, k, r, s, st, pad)
    p, q = oracle.conv_out_dims(shp)
    x, wt, dy = _inputs(shp, 13, scale=3.0)
    X = np.array(_hv(x), dtype=object).reshape(n, h, w, c)
    Wt = np.array(_hv(wt), dtype=object).reshape(k, r, s, c)
    DY = np.array(_hv(dy), dtype=object).reshape(n, p, q, k)
    cp, kp = (c + 7) // 8 * 8, (k + 7) // 8 * 8

    def xat(b, i, j, ch):
        return X[b, i, j, ch] if 0 <= i < h and 0 <= j < w and ch < c else Fraction(0)

    # forward: the im2col row of (b, i, j) against filter row kk, columns (r, s, c < Cp)
    got = oracle.conv_fwd_f16acc(shp, x, wt).view(np.uint16)
    for b in range(n):
        for i in range(p):
            for j in range(q):
                col = [xat(b, i * st - pad + rr, j * st - pad + ss, ch)
                       for rr in range(r) for ss in range(s) for ch in range(cp)]
                for kk in range(k):
                    wrow = [Wt[kk, rr, ss, ch] if ch < c else Fraction(0)
                            for rr in range(r) for ss in range(s) for ch in range(cp)]
                    want = _blocks16([a * bb for a, bb in zip(col, wrow)])
                    assert int(got[b, i, j, kk]) == want, ("fwd", b, i, j, kk)

    # data gradient: enumerate every forward term x[b, hh, ww, cc] * W[kk, rr, ss, cc]
    # that touches (hh, ww); the declared order is taps by decreasing (r, s)
    # among those that reach the position (whether or not their source lies on
    # the output grid), then output channels k < Kp
    got = oracle.conv_dgrad_f16acc(shp, dy, wt).view(np.uint16)
    for b in range(n):
        for hh in range(h):
            for ww in range(w):
                taps = [(rr, ss) for rr in range(r) for ss in range(s)
                        if (hh + pad - rr) % st == 0 and (ww + pad - ss) % st == 0]
                taps.sort(reverse=True)
                for cc in range(c):
                    terms = []
                    for rr, ss in taps:
                        pi, qj = (hh + pad - rr) // st, (ww + pad - ss) // st
                        on = 0 <= pi < p and 0 <= qj < q and hh + pad - rr >= 0 and ww + pad - ss >= 0
                        for kk in range(kp):
                            terms.append(DY[b, pi, qj, kk] * Wt[kk, rr, ss, cc]
                                         if on and kk < k else Fraction(0))
                    assert int(got[b, hh, ww, cc]) == _blocks16(terms), ("dgrad", b, hh, ww, cc)

    # weight gradient: pixels (b, i, j) in order
    got = oracle.conv_wgrad_f16acc(shp, x, dy).view(np.uint16)
    for kk in range(k):
        for rr in range(r):
            for ss in range(s):
                for cc in range(c):
                    terms = [DY[b, i, j, kk] * xat(b, i * st - pad + rr, j * st - pad + ss, cc)
                             for b in range(n) for i in range(p) for j in range(q)]
                    assert int(got[kk, rr, ss, cc]) == _blocks16(terms), ("wgrad", kk, rr, ss, cc)


def test_binary16_accumulation_costs_accuracy():
    # sanity of the study: on a 3x3 layer with a 1152-long reduction the
    # binary16 accumulator is further from the exact sums than one rounding
    shp = oracle.conv_shape(2, 128, 8, 8, 16, 3, 3, 1, 1)
    x, w, _ = _inputs(shp, 14)
    y64, y16 = oracle.conv_fwd(shp, x, w)
    ys = oracle.conv_fwd_f16acc(shp, x, w).astype(np.float64)
    e_def = np.sqrt(np.mean((y16.astype(np.float64) - y64) ** 2))
    e_str = np.sqrt(np.mean((ys - y64) ** 2))
    assert e_str > 2 * e_def
