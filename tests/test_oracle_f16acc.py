"""Pins for the oracle's strict binary16 arithmetic (all operations in FP16,
the literal reading of Section 5.2), used to measure what the float32
accumulators of the default path buy.

- fma16: exact rational evaluation (tests/exact.py) of round(a*b + c) on
  random and constructed binary16 triples, including subnormals, overflow
  and halfway cases.
- SGD with binary16 arithmetic: exact rational evaluation of the three
  fused multiply-adds with binary16 scalars; one hand-derived example where
  the extra rounding of d changes the momentum by one ulp.
- Convolutions as chains of binary16 fmas (one rounding per term, in a
  declared order, padding taps not terms):
  (a) a reduction of one term is one rounding of one product, equal to the
      (separately pinned) single rounding of the exact sum;
  (b) on small-integer data every partial sum is a binary16 integer, so the
      result is exact;
  (c) hand-derived values: 4,096 terms of 1.0 stagnate at 2048 (2048 + 1 is
      a tie and rounds to even), and 1 + 2^-11 + 2^-11 taken in channel
      order stays 1 while the exact sum 1 + 2^-10 is representable;
  (d) an independent brute force on tiny shapes: the terms of each output
      enumerated from the index formulas of Section 5.1's convolutions,
      sorted by the declared key, and chained in exact rational arithmetic
      with one binary16 rounding per term (signed zeros by the IEEE rules).
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


def _fma_bits(a, b, c):
    """binary16 bits of round(a*b + c) from exact rationals, with the IEEE
    sign of an exact zero (+0 unless the product and c are both -0)."""
    q = half_value(a) * half_value(b) + half_value(c)
    if q == 0:
        prod_neg = (a ^ b) & 0x8000
        return 0x8000 if (prod_neg and (c & 0x8000) and half_value(c) == 0) else 0
    return to_half_bits(q)


def _chain(pairs):
    acc = 0x0000
    for a, b in pairs:
        acc = _fma_bits(a, b, acc)
    return acc


@pytest.mark.parametrize("shape", [(1, 1, 4, 4, 1, 1, 1, 1, 0), (1, 1, 5, 5, 1, 1, 1, 2, 0)])
def test_one_term_is_one_rounding(shape):
    # C = K = R = S = N*P*Q... = 1 term per output: fma16(a, b, +0) = RNE16(a*b)
    n, c, h, w, k, r, s, st, pad = shape
    shp = oracle.conv_shape(n, c, h, w, k, r, s, st, pad)
    x, wt, dy = _inputs(shp, 11)
    assert np.array_equal(oracle.conv_fwd_f16acc(shp, x, wt).view(np.uint16),
                          oracle.conv_fwd(shp, x, wt)[1].view(np.uint16))
    assert np.array_equal(oracle.conv_dgrad_f16acc(shp, dy, wt).view(np.uint16),
                          oracle.conv_dgrad(shp, dy, wt)[1].view(np.uint16))
    shp1 = oracle.conv_shape(1, 3, 1, 1, 2, 1, 1)
    x1, _, dy1 = _inputs(shp1, 12)
    assert np.array_equal(oracle.conv_wgrad_f16acc(shp1, x1, dy1).view(np.uint16),
                          oracle.conv_wgrad(shp1, x1, dy1)[1].view(np.uint16))


def test_stagnation_worked_example():
    # 4,096 channels of x = 1, w = 1: the chain reaches 2048, where the
    # binary16 spacing is 2, so 2048 + 1 is a tie that rounds to even (2048)
    # and every further term is lost.  One rounding of the exact sum gives
    # 4096.  (A 16-term block accumulator would reach 4096 exactly.)
    shp = oracle.conv_shape(1, 4096, 1, 1, 1, 1, 1)
    x = np.ones((1, 1, 1, 4096), np.float16)
    w = np.ones((1, 1, 1, 4096), np.float16)
    assert int(oracle.conv_fwd_f16acc(shp, x, w).view(np.uint16)[0, 0, 0, 0]) == 0x6800
    assert float(oracle.conv_fwd(shp, x, w)[1][0, 0, 0, 0]) == 4096.0
    # the same through the weight gradient: 4,096 pixels of dy = x = 1
    shpw = oracle.conv_shape(1, 1, 64, 64, 1, 1, 1)
    ones = np.ones((1, 64, 64, 1), np.float16)
    assert int(oracle.conv_wgrad_f16acc(shpw, ones, ones).view(np.uint16).reshape(-1)[0]) == 0x6800
    # and the data gradient: 4,096 output channels
    shpd = oracle.conv_shape(1, 1, 1, 1, 4096, 1, 1)
    assert int(oracle.conv_dgrad_f16acc(shpd, np.ones((1, 1, 1, 4096), np.float16),
                                        np.ones((4096, 1, 1, 1), np.float16))
               .view(np.uint16).reshape(-1)[0]) == 0x6800


def test_order_worked_example():
    # channels (1, 2^-11, 2^-11) against w = 1: 1 + 2^-11 is a tie between 1
    # and 1 + 2^-10 and rounds to even (1), twice; the exact sum 1 + 2^-10
    # (0x3C01) is what one rounding gives.  With the channels in the other
    # order the chain reaches it too: the order is part of the definition.
    shp = oracle.conv_shape(1, 3, 1, 1, 1, 1, 1)
    w = np.ones((1, 1, 1, 3), np.float16)
    x = np.array([1.0, 2.0 ** -11, 2.0 ** -11], np.float16).reshape(1, 1, 1, 3)
    assert int(oracle.conv_fwd_f16acc(shp, x, w).view(np.uint16).reshape(-1)[0]) == 0x3C00
    assert int(oracle.conv_fwd(shp, x, w)[1].view(np.uint16).reshape(-1)[0]) == 0x3C01
    xr = x[..., ::-1].copy()
    assert int(oracle.conv_fwd_f16acc(shp, xr, w).view(np.uint16).reshape(-1)[0]) == 0x3C01


def test_signed_zero_and_padding_are_not_terms():
    # a single tiny negative product rounds to -0; a padding tap after it is
    # not a term, so -0 stays (a +0 term would turn it into +0)
    shp = oracle.conv_shape(1, 1, 1, 2, 1, 1, 3, 1, (0, 1))   # W = 2, S = 3, pad 1 along w
    x = np.array([2.0 ** -24, 0.0], np.float16).reshape(1, 1, 2, 1)
    w = np.array([0.0, -0.25, 0.0], np.float16).reshape(1, 1, 3, 1)
    y = oracle.conv_fwd_f16acc(shp, x, w).view(np.uint16).reshape(-1)
    # q = 0: taps s = 1 (x[0] * -0.25 = -2^-26 -> -0), s = 2 (x[1] = 0 times +0 = +0: -0 + +0 = +0)
    assert int(y[0]) == 0x0000
    # q = 1: taps s = 0 (x[0] * +0 = +0), s = 1 (x[1] = +0 * -0.25 = -0: +0 + -0 = +0), s = 2 padding
    assert int(y[1]) == 0x0000
    x2 = np.array([0.0, 2.0 ** -24], np.float16).reshape(1, 1, 2, 1)
    # q = 1: s = 0: +0*+0 = +0; s = 1: 2^-24 * -0.25 -> -0: +0 + -2^-26 rounds to -0;
    # s = 2 lies in the padding and is not a term, so -0 remains
    assert int(oracle.conv_fwd_f16acc(shp, x2, w).view(np.uint16).reshape(-1)[1]) == 0x8000


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


def _bits(a):
    return np.ascontiguousarray(a).view(np.uint16)


@pytest.mark.parametrize("shape", [(1, 3, 5, 5, 4, 3, 3, 1, 1), (2, 8, 6, 5, 3, 3, 3, 2, 1),
                                   (1, 5, 7, 7, 2, 3, 3, 2, 0), (1, 16, 4, 4, 8, 1, 1, 2, 0),
                                   (1, 2, 9, 9, 3, 7, 7, 2, 3)])
def test_brute_force_chain_order(shape):
    n, c, h, w, k, r, s, st, pad = shape
    shp = oracle.conv_shape(n, c, h, w, k, r, s, st, pad)
    p, q = oracle.conv_out_dims(shp)
    x, wt, dy = _inputs(shp, 13, scale=3.0)
    X, Wt, DY = _bits(x), _bits(wt), _bits(dy)

    # forward: every (r, s, c) whose position lies in the image, keyed (r, s, c)
    got = _bits(oracle.conv_fwd_f16acc(shp, x, wt))
    for b in range(n):
        for i in range(p):
            for j in range(q):
                for kk in range(k):
                    terms = []
                    for rr in range(r):
                        for ss in range(s):
                            hi, wj = i * st - pad + rr, j * st - pad + ss
                            if 0 <= hi < h and 0 <= wj < w:
                                terms += [((rr, ss, ch), int(X[b, hi, wj, ch]), int(Wt[kk, rr, ss, ch]))
                                          for ch in range(c)]
                    terms.sort(key=lambda t: t[0])
                    want = _chain([(a_, b_) for _, a_, b_ in terms])
                    assert int(got[b, i, j, kk]) == want, ("fwd", b, i, j, kk)

    # data gradient: every forward term x[b, hh, ww, cc] * W[kk, rr, ss, cc] that
    # lands on an output grid point, keyed (r, s, k)
    got = _bits(oracle.conv_dgrad_f16acc(shp, dy, wt))
    for b in range(n):
        for hh in range(h):
            for ww in range(w):
                for cc in range(c):
                    terms = []
                    for i in range(p):
                        for j in range(q):
                            rr, ss = hh - (i * st - pad), ww - (j * st - pad)
                            if 0 <= rr < r and 0 <= ss < s:
                                terms += [((rr, ss, kk), int(DY[b, i, j, kk]), int(Wt[kk, rr, ss, cc]))
                                          for kk in range(k)]
                    terms.sort(key=lambda t: t[0])
                    want = _chain([(a_, b_) for _, a_, b_ in terms])
                    assert int(got[b, hh, ww, cc]) == want, ("dgrad", b, hh, ww, cc)

    # weight gradient: output pixels (b, i, j) in order, in-image taps only
    got = _bits(oracle.conv_wgrad_f16acc(shp, x, dy))
    for kk in range(k):
        for rr in range(r):
            for ss in range(s):
                for cc in range(c):
                    pairs = [(int(DY[b, i, j, kk]), int(X[b, i * st - pad + rr, j * st - pad + ss, cc]))
                             for b in range(n) for i in range(p) for j in range(q)
                             if 0 <= i * st - pad + rr < h and 0 <= j * st - pad + ss < w]
                    assert int(got[kk, rr, ss, cc]) == _chain(pairs), ("wgrad", kk, rr, ss, cc)


def test_any_layout_same_values():
    # the order is declared in logical indices, so NCHW gives the same values
    shp = oracle.conv_shape(2, 6, 5, 5, 4, 3, 3, 2, 1)
    shq = oracle.conv_shape(2, 6, 5, 5, 4, 3, 3, 2, 1, layout="NCHW")
    x, wt, dy = _inputs(shp, 15)
    xn, wn, dyn = x.transpose(0, 3, 1, 2).copy(), wt.transpose(0, 3, 1, 2).copy(), dy.transpose(0, 3, 1, 2).copy()
    assert np.array_equal(_bits(oracle.conv_fwd_f16acc(shp, x, wt)).transpose(0, 3, 1, 2),
                          _bits(oracle.conv_fwd_f16acc(shq, xn, wn)))
    assert np.array_equal(_bits(oracle.conv_dgrad_f16acc(shp, dy, wt)).transpose(0, 3, 1, 2),
                          _bits(oracle.conv_dgrad_f16acc(shq, dyn, wn)))
    assert np.array_equal(_bits(oracle.conv_wgrad_f16acc(shp, x, dy)).transpose(0, 3, 1, 2),
                          _bits(oracle.conv_wgrad_f16acc(shq, xn, dyn)))


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


def test_sampled_entry_points_equal_full():
    shp = oracle.conv_shape(2, 12, 7, 7, 10, 3, 3, 2, 1)
    x, wt, dy = _inputs(shp, 16)
    for full, at, a, b in ((oracle.conv_fwd_f16acc, oracle.conv_fwd_f16acc_at, x, wt),
                           (oracle.conv_dgrad_f16acc, oracle.conv_dgrad_f16acc_at, dy, wt),
                           (oracle.conv_wgrad_f16acc, oracle.conv_wgrad_f16acc_at, x, dy)):
        f = _bits(full(shp, a, b)).reshape(-1)
        idx = np.arange(0, f.size, 3, dtype=np.int64)
        assert np.array_equal(_bits(at(shp, a, b, idx)), f[idx])
