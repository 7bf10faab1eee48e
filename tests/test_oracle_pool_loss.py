"""Pins of the oracle's pooling and loss definitions (the parts of ResNet-50
around the residual blocks, Section 5.1) against references that share
nothing with it: numpy sliding windows and scipy's maximum filter for max
pooling, closed forms and numpy means for average pooling, scipy's
logsumexp and finite differences for the softmax cross-entropy, and exact
rational rounding (tests/exact.py) wherever a value is rounded to binary16."""

from fractions import Fraction

import numpy as np
import pytest
from numpy.lib.stride_tricks import sliding_window_view
from scipy import ndimage, special

import oracle
from exact import to_half
from paper_1911_07384_amd import synth


def _half_of(v: float) -> float:
    return float(to_half(Fraction(v)))


def _rne16_exact(a):
    """binary16 rounding of float64 values by exact rational arithmetic."""
    return np.array([_half_of(float(v)) for v in np.ravel(a)], np.float64).reshape(np.shape(a))


def _nhwc(x_nchw):
    return np.ascontiguousarray(np.transpose(x_nchw, (0, 2, 3, 1)))


# ---- max pooling ---------------------------------------------------------------

POOLS = [  # n, c, h, w, r, stride, pad
    (2, 3, 9, 9, 3, 2, 1),     # ResNet-50 stem pool geometry, small
    (1, 4, 8, 7, 3, 2, 1),     # even / odd sizes
    (2, 2, 6, 6, 2, 2, 0),
    (1, 3, 5, 5, 3, 1, 1),
    (1, 1, 4, 4, 3, 3, 1),     # windows that overhang the far edge
]


def _window_ref(x_nchw, r, stride, pad):
    """Max and first argmax of every window, via -inf padding and numpy views."""
    xp = np.pad(x_nchw.astype(np.float64), ((0, 0), (0, 0), (pad, pad), (pad, pad)),
                constant_values=-np.inf)
    win = sliding_window_view(xp, (r, r), axis=(2, 3))[:, :, ::stride, ::stride]
    flat = win.reshape(win.shape[:4] + (r * r,))
    return flat.max(axis=-1), flat.argmax(axis=-1)


@pytest.mark.parametrize("case", POOLS)
@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
def test_maxpool_fwd_matches_window_max(case, layout):
    n, c, h, w, r, st, pad = case
    x = synth.normal_f16((n, c, h, w), 1.0, 3, 1)
    # exact ties, so the first-position rule is exercised
    x = (np.round(x.astype(np.float64) * 2) / 2).astype(np.float16)
    shp = oracle.pool_shape(n, c, h, w, r, r, st, pad, layout)
    y, idx = oracle.maxpool_fwd(shp, _nhwc(x) if layout == "NHWC" else x)
    ref, arg = _window_ref(x, r, st, pad)
    if layout == "NHWC":
        ref, arg = np.transpose(ref, (0, 2, 3, 1)), np.transpose(arg, (0, 2, 3, 1))
    assert y.shape == ref.shape
    np.testing.assert_array_equal(y.astype(np.float64), ref)
    np.testing.assert_array_equal(idx, arg)


def test_maxpool_stride1_equals_scipy_maximum_filter():
    x = synth.normal_f16((1, 2, 10, 11), 1.0, 4, 1)
    shp = oracle.pool_shape(1, 2, 10, 11, 3, 3, 1, 1, "NCHW")
    y, _ = oracle.maxpool_fwd(shp, x)
    ref = ndimage.maximum_filter(x.astype(np.float64), size=(1, 1, 3, 3), mode="constant",
                                 cval=-np.inf)
    np.testing.assert_array_equal(y.astype(np.float64), ref)


def test_maxpool_nan_propagates_and_wins():
    x = np.zeros((1, 1, 3, 3), np.float16)
    x[0, 0, 1, 1] = np.nan
    x[0, 0, 2, 2] = np.nan
    x[0, 0, 0, 0] = 5
    shp = oracle.pool_shape(1, 1, 3, 3, 3, 3, 1, 0, "NCHW")
    y, idx = oracle.maxpool_fwd(shp, x)
    assert np.isnan(y[0, 0, 0, 0]) and idx[0, 0, 0, 0] == 4  # the first NaN in scan order


def test_maxpool_negative_zero_tie_keeps_first():
    x = np.array([-0.0, 0.0, -1.0, -2.0], np.float16).reshape(1, 1, 2, 2)
    shp = oracle.pool_shape(1, 1, 2, 2, 2, 2, 1, 0, "NCHW")
    y, idx = oracle.maxpool_fwd(shp, x)
    assert idx[0, 0, 0, 0] == 0 and np.signbit(y[0, 0, 0, 0])


@pytest.mark.parametrize("case", POOLS)
def test_maxpool_bwd_is_the_adjoint_of_the_selection(case):
    # With small-integer dy every sum is exact, so the adjoint identity and the
    # conservation of the gradient hold exactly.
    n, c, h, w, r, st, pad = case
    x = synth.normal_f16((n, c, h, w), 1.0, 5, 1)
    shp = oracle.pool_shape(n, c, h, w, r, r, st, pad, "NCHW")
    _, arg = _window_ref(x, r, st, pad)
    p, q = arg.shape[2:]
    rng = np.random.default_rng(0)
    dy = rng.integers(-8, 9, (n, c, p, q)).astype(np.float16)
    dx = oracle.maxpool_bwd(shp, x, dy).astype(np.float64)
    # scatter of dy to the winning positions, written independently
    ref = np.zeros((n, c, h, w))
    for i0 in range(n):
        for i1 in range(c):
            for i2 in range(p):
                for i3 in range(q):
                    t = arg[i0, i1, i2, i3]
                    ref[i0, i1, i2 * st - pad + t // r, i3 * st - pad + t % r] += dy[i0, i1, i2, i3]
    np.testing.assert_array_equal(dx, ref)
    assert dx.sum() == dy.astype(np.float64).sum()
    xp = rng.integers(-4, 5, x.shape).astype(np.float64)
    ysel = np.take_along_axis(
        sliding_window_view(np.pad(xp, ((0, 0), (0, 0), (pad, pad), (pad, pad))), (r, r),
                            axis=(2, 3))[:, :, ::st, ::st].reshape(n, c, p, q, r * r),
        arg[..., None], axis=-1)[..., 0]
    assert np.sum(ysel * dy) == np.sum(xp * dx)


def test_maxpool_bwd_rounds_the_sum_once():
    # two windows select the same position: 1 + 2^-11 is not binary16, the
    # exact sum rounds to 1 (tie to even), while the parts are exact
    x = np.array([[0, 9, 0]], np.float16).reshape(1, 1, 1, 3)
    shp = oracle.pool_shape(1, 1, 1, 3, 1, 2, (1, 1), (0, 0), "NCHW")
    dy = np.array([1.0, 2.0 ** -11], np.float16).reshape(1, 1, 1, 2)
    dx = oracle.maxpool_bwd(shp, x, dy)
    assert dx[0, 0, 0, 1] == np.float16(1.0)


# ---- global average pooling ------------------------------------------------------

def test_avgpool_constant_is_exact():
    x = np.full((2, 7, 7, 5), 0.3, np.float16)
    shp = oracle.pool_shape(2, 5, 7, 7, 7, 7, 1, 0, "NHWC")
    y64, y = oracle.avgpool_fwd(shp, x)
    assert np.all(y == x[0, 0, 0, 0]) and np.all(y64 == float(x[0, 0, 0, 0]))


@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
def test_avgpool_matches_numpy_mean(layout):
    x = synth.normal_f16((3, 6, 7, 7), 1.0, 6, 1)
    shp = oracle.pool_shape(3, 6, 7, 7, 7, 7, 1, 0, layout)
    y64, y = oracle.avgpool_fwd(shp, _nhwc(x) if layout == "NHWC" else x)
    # the exact mean as a rational, then exact rounding
    exact = np.array([[float(to_half(sum(Fraction(float(v)) for v in x[i, j].ravel()) / 49))
                       for j in range(6)] for i in range(3)])
    np.testing.assert_array_equal(y.astype(np.float64), exact)
    np.testing.assert_allclose(y64, x.astype(np.float64).mean(axis=(2, 3)), rtol=1e-15)


def test_avgpool_bwd_closed_form_and_adjoint():
    rng = np.random.default_rng(1)
    dy = (rng.integers(-20, 21, (2, 4)) * 49 / 1024).astype(np.float16)  # divisible by 49
    shp = oracle.pool_shape(2, 4, 7, 7, 7, 7, 1, 0, "NHWC")
    dx = oracle.avgpool_bwd(shp, dy).astype(np.float64)
    np.testing.assert_array_equal(dx, np.broadcast_to(dy.astype(np.float64)[:, None, None, :] / 49,
                                                      dx.shape))
    x = rng.integers(-3, 4, (2, 7, 7, 4)).astype(np.float16)
    y64, _ = oracle.avgpool_fwd(shp, x)
    assert abs(np.sum(y64 * dy) - np.sum(x.astype(np.float64) * dx)) < 1e-12


def test_avgpool_bwd_rounds_the_quotient():
    dy = np.array([[1.0]], np.float16)
    shp = oracle.pool_shape(1, 1, 7, 7, 7, 7, 1, 0, "NHWC")
    dx = oracle.avgpool_bwd(shp, dy)
    assert float(dx[0, 0, 0, 0]) == _half_of(1 / 49)


# ---- classifier bias and softmax cross-entropy ---------------------------------------

def _logits(z, b):
    """binary16 logits l = rne16(z + b) by exact rational rounding."""
    return np.array([[float(to_half(Fraction(float(z[i, j])) + Fraction(float(b[j]))))
                      for j in range(z.shape[1])] for i in range(z.shape[0])])


def test_softmax_ce_uniform_closed_form():
    n, k = 4, 10
    out = oracle.softmax_ce(np.zeros((n, k), np.float16), np.zeros(k, np.float16), [0, 3, 9, 3])
    assert abs(out["loss"] - np.log(k)) < 1e-15
    dz = out["dz"].astype(np.float64)
    lab = np.array([0, 3, 9, 3])
    ref = np.full((n, k), _half_of(1 / (k * n)))
    ref[np.arange(n), lab] = _half_of((1 / k - 1) / n)
    np.testing.assert_array_equal(dz, ref)
    # db sums the stored column entries exactly
    np.testing.assert_array_equal(out["db"].astype(np.float64), _rne16_exact(ref.sum(axis=0)))


def test_softmax_ce_matches_scipy_and_finite_differences():
    n, k = 6, 37
    z = synth.normal_f16((n, k), 3.0, 7, 1)
    b = synth.normal_f16((k,), 0.5, 7, 2)
    lab = synth.labels(n, k, 7, 3)
    out = oracle.softmax_ce(z, b, lab)
    l = _logits(z, b)
    rows = special.logsumexp(l, axis=1) - l[np.arange(n), lab]
    np.testing.assert_allclose(out["loss_rows"], rows, rtol=1e-14, atol=1e-14)
    assert abs(out["loss"] - rows.mean()) < 1e-14

    def mean_loss(lv):
        return np.mean(special.logsumexp(lv, axis=1) - lv[np.arange(n), lab])

    g = np.zeros_like(l)
    h = 1e-6
    for i in range(n):
        for j in range(k):
            lp, lm = l.copy(), l.copy()
            lp[i, j] += h
            lm[i, j] -= h
            g[i, j] = (mean_loss(lp) - mean_loss(lm)) / (2 * h)
    dz = out["dz"].astype(np.float64)
    # the stored gradient is the derivative rounded once to binary16
    assert np.all(np.abs(dz - g) <= 2.0 ** -11 * np.abs(g) + 2.0 ** -24 + 1e-9)
    # rows of the unrounded gradient sum to zero; the rounded ones nearly
    assert np.all(np.abs(dz.sum(axis=1)) <= k * 2.0 ** -11 * np.abs(dz).max())


def test_softmax_ce_large_logits_do_not_overflow():
    z = np.array([[60000.0, 0.0, -60000.0], [65504.0, 65504.0, 65504.0]], np.float16)
    b = np.zeros(3, np.float16)
    out = oracle.softmax_ce(z, b, [0, 1])
    assert np.isfinite(out["loss"])
    assert out["loss_rows"][0] == 0.0 and abs(out["loss_rows"][1] - np.log(3)) < 1e-15
    assert out["dz"][0, 0] == 0.0 and out["dz"][0, 1] == 0.0


def test_softmax_ce_bias_rounding_is_one_binary16_rounding():
    # z + b = 1 + 2^-11 is a tie between 1 and 1 + 2^-10: rounds to 1 (even)
    z = np.array([[1.0, 0.0]], np.float16)
    b = np.array([2.0 ** -11, 0.0], np.float16)
    out = oracle.softmax_ce(z, b, [1])
    ref = special.logsumexp([1.0, 0.0]) - 0.0
    assert abs(out["loss_rows"][0] - ref) < 1e-15


def test_softmax_ce_gradient_of_full_batch_is_subnormal():
    # ResNet-50's 1000 classes at batch 128: the non-label entries of the
    # gradient sit near 1/(1000*128), inside the binary16 subnormal range, and
    # must not be flushed to zero
    n, k = 128, 1000
    z = synth.normal_f16((n, k), 0.01, 8, 1)
    out = oracle.softmax_ce(z, np.zeros(k, np.float16), synth.labels(n, k, 8, 2))
    a = np.abs(out["dz"].astype(np.float64))
    assert np.mean((a > 0) & (a < 2.0 ** -14)) > 0.99
    assert np.all(a > 0)
