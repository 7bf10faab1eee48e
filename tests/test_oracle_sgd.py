"""Pins for the oracle's momentum-SGD step (FP16 weights and momentum, no
master copy; Section 5.1 recipe, Section 5.2).

The declared float32 sequence is  d = fma(wd, w, g);  m' = rne16(fma(mu, m, d));
w' = rne16(fma(-lr, m', w)).  It is pinned by (a) hand-derived worked
examples, (b) an exact rational evaluation of the same sequence, (c) a closed
form for constant gradients where every step is exact.
"""

from fractions import Fraction

import numpy as np
import pytest

import oracle
from exact import INF, half_value, to_half, to_half_bits, to_single

F = Fraction


def f32(x) -> Fraction:
    return F(float(np.float32(x)))


def exact_sgd(wb, gb, mb, lr, mom, wd):
    """Exact-rational evaluation of the declared sequence on binary16 inputs."""
    w, g, m = half_value(wb), half_value(gb), half_value(mb)
    lr, mom, wd = f32(lr), f32(mom), f32(wd)
    d = to_single(wd * w + g)
    m1q = to_single(mom * m + d)
    m1 = to_half_bits(m1q) if abs(m1q) != INF else (0x7C00 if m1q > 0 else 0xFC00)
    m1v = half_value(m1)
    if abs(m1v) == INF:
        wq = -m1v if lr > 0 else m1v
        return m1, (0x7C00 if wq > 0 else 0xFC00)
    wq = to_single(-lr * m1v + w)
    w1 = to_half_bits(wq) if abs(wq) != INF else (0x7C00 if wq > 0 else 0xFC00)
    return m1, w1


# (w, g, m, lr, momentum, wd) -> (m', w'), hand derived:
#  basic: d = 0.5, m' = 0.5; w' = 1 - 0.1f*0.5 = 0.94999999 -> nearest binary16 0.9501953125.
#  wd=1e-4: the decay term (1e-4) is below half an ulp of m' = 0.5 in binary16.
#  m=0.25: fl32(0.9f*0.25 + 0.5) = 0.72500002; binary16 0.72509765625 (0x39CD);
#          w' = 1 - 0.1f*0.72509765625 = 0.92749017 -> 0.927734375 (0x3B6C).
#  stagnation: lr*|m'| = 2^-14 * 0.035 ~ 2.1e-6 is below half an ulp of w (2^-17): w unchanged.
#  tie: w = 2048, m' = -1, w' = 2049 is the midpoint of 2048 and 2050 -> 2048 (even).
#  overflow: m' = -400 (0xDE40); w' = 65504 + 40 = 65544 >= 65520 -> +inf.
#  subnormal: m' = 2^-10 (0x1400); w' = 2^-20 - 2^-14 = -1008 * 2^-24 (0x83F0).
WORKED = [
    ((0x3C00, 0x3800, 0x0000, 0.1, 0.9, 0.0), (0x3800, 0x3B9A)),
    ((0x3C00, 0x3800, 0x0000, 0.1, 0.9, 1e-4), (0x3800, 0x3B9A)),
    ((0x3C00, 0x3800, 0x3400, 0.1, 0.9, 0.0), (0x39CD, 0x3B6C)),
    ((0x278D, 0x287B, 0x0000, 2.0 ** -14, 0.9, 1e-4), (0x287B, 0x278D)),
    ((0x6800, 0xBC00, 0x0000, 1.0, 0.9, 0.0), (0xBC00, 0x6800)),
    ((0x7BFF, 0xDE40, 0x0000, 0.1, 0.9, 0.0), (0xDE40, 0x7C00)),
    ((0x0010, 0x1400, 0x0000, 2.0 ** -4, 0.9, 1e-4), (0x1400, 0x83F0)),
]


@pytest.mark.parametrize("inp,want", WORKED)
def test_worked_examples(inp, want):
    wb, gb, mb, lr, mom, wd = inp
    w1, m1 = oracle.sgd_f32(np.array([wb], np.uint16), np.array([gb], np.uint16),
                            np.array([mb], np.uint16), lr, mom, wd)
    got = (int(m1.view(np.uint16)[0]), int(w1.view(np.uint16)[0]))
    assert got == want, [hex(v) for v in got]
    assert exact_sgd(wb, gb, mb, lr, mom, wd) == want


def _finite_halves(rng, n, max_exp=14):
    """Random finite binary16 bit patterns, including subnormals and zeros."""
    b = rng.integers(0, 1 << 15, size=n).astype(np.uint16)
    exp = (b >> 10) & 31
    b = np.where(exp > max_exp + 15, b & 0x83FF | np.uint16((max_exp + 15) << 10), b)
    sign = (rng.random(n) < 0.5).astype(np.uint16) << 15
    return (b | sign).astype(np.uint16)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_against_exact(seed):
    rng = np.random.default_rng(seed)
    n = 1500
    w = _finite_halves(rng, n)
    g = _finite_halves(rng, n)
    m = _finite_halves(rng, n)
    lr = float(rng.choice([0.1, 2.0 ** -14, 1.0, 0.0125]))
    mom = float(rng.choice([0.9, 0.0, 0.99]))
    wd = float(rng.choice([1e-4, 0.0, 5e-5]))
    w1, m1 = oracle.sgd_f32(w, g, m, lr, mom, wd)
    w1, m1 = w1.view(np.uint16), m1.view(np.uint16)
    for i in range(n):
        em, ew = exact_sgd(int(w[i]), int(g[i]), int(m[i]), lr, mom, wd)
        assert (int(m1[i]), int(w1[i])) == (em, ew), (i, hex(w[i]), hex(g[i]), hex(m[i]))


@pytest.mark.parametrize("fn", [oracle.sgd_f32, oracle.sgd_f64])
def test_constant_gradient_closed_form(fn):
    # g = 2^-4, mu = 1/2, wd = 0, lr = 2^-3, w0 = 1, m0 = 0:
    # m_k = 2 g (1 - 2^-k);  w_k = 1 - lr * sum_{j<=k} m_j = 1 - 2^-6 (k - 1 + 2^-k),
    # all exactly representable in binary16 for k <= 5, so both variants must
    # reproduce the closed form exactly.
    w = np.array([1.0], np.float16)
    m = np.array([0.0], np.float16)
    g = np.array([2.0 ** -4], np.float16)
    for k in range(1, 6):
        w, m = fn(w, g, m, 2.0 ** -3, 0.5, 0.0)
        assert float(m[0]) == 2 * 2.0 ** -4 * (1 - 2.0 ** -k)
        assert float(w[0]) == 1 - 2.0 ** -6 * (k - 1 + 2.0 ** -k)


def test_f64_variant_differs_only_by_intermediate_rounding():
    # the float64 variant rounds only at m and w; on random data it agrees
    # with the float32 sequence except where float32 intermediates land on
    # the other side of a binary16 rounding boundary (rare)
    rng = np.random.default_rng(5)
    n = 20000
    w = rng.normal(0, 0.05, n).astype(np.float16)
    g = rng.normal(0, 0.01, n).astype(np.float16)
    m = rng.normal(0, 0.01, n).astype(np.float16)
    a = oracle.sgd_f32(w, g, m, 0.1, 0.9, 1e-4)
    b = oracle.sgd_f64(w, g, m, 0.1, 0.9, 1e-4)
    diff = np.mean(a[0].view(np.uint16) != b[0].view(np.uint16))
    assert diff < 0.01
