"""Pins for the oracle's convolutions (ResNet-50 convolutions, Section 5.1;
FP16 storage with one rounding at the store, Section 5.2).

(1) brute-force im2col + a numpy float64 matrix product on tiny shapes;
(2) the adjoint identities <dy, fwd(x;W)> = <dgrad(dy;W), x> = <wgrad(x,dy), W>;
(3) delta filters reproduce (shifted) inputs bit-exactly;
(4) a one-hot dy gives dx = a scattered filter slice and dW = an input patch;
(5) the sampled entry points agree with the full passes;
(6) the stored binary16 equals numpy's rounding of the float64 sums.
"""

import itertools

import numpy as np
import pytest

import oracle
from paper_1911_07384_amd import synth


def _shapes():
    out = []
    for (n, c, k, hw, r, st) in [
        (1, 1, 1, 1, 1, 1), (2, 3, 8, 5, 3, 1), (1, 8, 3, 7, 3, 2), (2, 3, 3, 7, 7, 2),
        (1, 8, 8, 6, 1, 2), (2, 1, 8, 4, 3, 1), (1, 3, 1, 7, 7, 1), (2, 8, 3, 3, 3, 2),
        (1, 3, 8, 2, 1, 1), (2, 8, 8, 7, 3, 1),
    ]:
        for pad in sorted({0, r // 2}):
            if hw + 2 * pad < r:
                continue
            out.append((n, c, hw, hw, k, r, r, st, pad))
    # non-square spatial size and mixed stride/pad
    out.append((1, 3, 5, 7, 4, 3, 3, 2, 1))
    out.append((2, 5, 7, 4, 3, 3, 1, 1, 1))
    return out


def _inputs(shp, seed=0):
    n, c, h, w, k, r, s = (int(v) for v in shp[:7])
    lay = int(shp[11])
    p, q = oracle.conv_out_dims(shp)
    xs = (n, h, w, c) if lay == 0 else (n, c, h, w)
    ys = (n, p, q, k) if lay == 0 else (n, k, p, q)
    ws = (k, r, s, c) if lay == 0 else (k, c, r, s)
    x = synth.normal_f16(xs, 1.0, seed, 1)
    wt = synth.normal_f16(ws, 0.5, seed, 2)
    dy = synth.normal_f16(ys, 1.0, seed, 3)
    return x, wt, dy


def _to_nchw(a, lay):
    return a if lay == 1 else np.moveaxis(a, -1, 1)


def _filter_to_kcrs(wt, lay):
    return wt if lay == 1 else np.transpose(wt, (0, 3, 1, 2))


def _im2col_conv(shp, x, wt):
    """Brute-force reference: explicit im2col matrix times the filter matrix."""
    n, c, h, w, k, r, s, sh, sw, ph, pw, lay = (int(v) for v in shp)
    p, q = oracle.conv_out_dims(shp)
    X = _to_nchw(x.astype(np.float64), lay)
    Wm = _filter_to_kcrs(wt.astype(np.float64), lay).reshape(k, c * r * s)
    cols = np.zeros((n * p * q, c * r * s))
    row = 0
    for ni in range(n):
        for pi in range(p):
            for qi in range(q):
                col = 0
                for ci in range(c):
                    for ri in range(r):
                        for si in range(s):
                            hh, ww = pi * sh - ph + ri, qi * sw - pw + si
                            if 0 <= hh < h and 0 <= ww < w:
                                cols[row, col] = X[ni, ci, hh, ww]
                            col += 1
                row += 1
    y = (cols @ Wm.T).reshape(n, p, q, k)  # NHWC
    return y if lay == 0 else np.moveaxis(y, -1, 1)


ALL = [(s, lay) for s in _shapes() for lay in ("NHWC", "NCHW")]


@pytest.mark.parametrize("sh,layout", ALL)
def test_fwd_matches_im2col(sh, layout):
    n, c, h, w, k, r, s, st, pad = sh
    shp = oracle.conv_shape(n, c, h, w, k, r, s, st, pad, layout)
    x, wt, _ = _inputs(shp)
    y64, y16 = oracle.conv_fwd(shp, x, wt)
    ref = _im2col_conv(shp, x, wt)
    assert y64.shape == ref.shape
    scale = max(1.0, np.abs(ref).max())
    assert np.max(np.abs(y64 - ref)) <= 1e-13 * scale
    # one rounding at the store, checked against numpy's independent rounding
    assert np.array_equal(y16.view(np.uint16), y64.astype(np.float16).view(np.uint16))


@pytest.mark.parametrize("sh,layout", ALL)
def test_adjoint_identities(sh, layout):
    n, c, h, w, k, r, s, st, pad = sh
    shp = oracle.conv_shape(n, c, h, w, k, r, s, st, pad, layout)
    x, wt, dy = _inputs(shp, seed=7)
    y64, _ = oracle.conv_fwd(shp, x, wt)
    dx64, dx16 = oracle.conv_dgrad(shp, dy, wt)
    dw64, dw16 = oracle.conv_wgrad(shp, x, dy)
    X, Wt, DY = (a.astype(np.float64) for a in (x, wt, dy))
    a = np.sum(DY * y64)
    b = np.sum(dx64 * X)
    cc = np.sum(dw64 * Wt)
    mag = np.sum(np.abs(DY * y64)) + 1e-300
    assert abs(a - b) <= 1e-12 * mag
    assert abs(a - cc) <= 1e-12 * mag
    # the same identity on the rounded outputs, within the binary16 rounding
    # of every term: |<dy,y16> - <dx16,x>| <= 2^-11 (sum|dy*y| + sum|dx*x|)
    y16 = oracle.conv_fwd(shp, x, wt)[1].astype(np.float64)
    lhs = np.sum(DY * y16)
    rhs = np.sum(dx16.astype(np.float64) * X)
    bound = 2.0 ** -11 * (np.sum(np.abs(DY * y64)) + np.sum(np.abs(dx64 * X))) + 1e-300
    assert abs(lhs - rhs) <= bound
    rhs_w = np.sum(dw16.astype(np.float64) * Wt)
    bound_w = 2.0 ** -11 * (np.sum(np.abs(DY * y64)) + np.sum(np.abs(dw64 * Wt))) + 1e-300
    assert abs(lhs - rhs_w) <= bound_w


@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("r,shift", [(1, (0, 0)), (3, (0, 0)), (3, (1, -1)), (7, (2, 3)), (3, (-1, 0))])
def test_delta_filter_is_exact_copy(layout, r, shift):
    n, c, h, w = 2, 5, 6, 7
    pad = r // 2
    shp = oracle.conv_shape(n, c, h, w, c, r, r, 1, pad, layout)
    x, _, _ = _inputs(shp, seed=3)
    Wk = np.zeros((c, c, r, r), np.float16)  # KCRS
    dr, ds = shift
    for ci in range(c):
        Wk[ci, ci, pad + dr, pad + ds] = 1.0
    wt = Wk if layout == "NCHW" else np.ascontiguousarray(np.transpose(Wk, (0, 2, 3, 1)))
    _, y16 = oracle.conv_fwd(shp, x, wt)
    X = _to_nchw(x, 1 if layout == "NCHW" else 0)
    Y = _to_nchw(y16, 1 if layout == "NCHW" else 0)
    want = np.zeros_like(X)
    for hh in range(h):
        for ww in range(w):
            sh_, sw_ = hh + dr, ww + ds
            if 0 <= sh_ < h and 0 <= sw_ < w:
                want[:, :, hh, ww] = X[:, :, sh_, sw_]
    assert np.array_equal(Y.view(np.uint16), want.view(np.uint16))


@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("r,st,pad", [(3, 1, 1), (3, 2, 1), (1, 2, 0), (7, 2, 3), (1, 1, 0)])
def test_one_hot_dy(layout, r, st, pad):
    n, c, h, w, k = 2, 3, 9, 8, 4
    shp = oracle.conv_shape(n, c, h, w, k, r, r, st, pad, layout)
    p, q = oracle.conv_out_dims(shp)
    x, wt, _ = _inputs(shp, seed=11)
    lay = 0 if layout == "NHWC" else 1
    for (n0, k0, p0, q0) in [(1, 2, p - 1, 0), (0, 0, 0, q - 1), (1, 3, p // 2, q // 2)]:
        DY = np.zeros((n, k, p, q), np.float16)
        DY[n0, k0, p0, q0] = 1.0
        dy = DY if lay == 1 else np.ascontiguousarray(np.moveaxis(DY, 1, -1))
        _, dx16 = oracle.conv_dgrad(shp, dy, wt)
        _, dw16 = oracle.conv_wgrad(shp, x, dy)
        DX = _to_nchw(dx16, lay)
        DW = _filter_to_kcrs(dw16, lay)
        Wk = _filter_to_kcrs(wt, lay)
        X = _to_nchw(x, lay)
        want_dx = np.zeros((n, c, h, w), np.float16)
        want_dw = np.zeros((k, c, r, r), np.float16)
        for ri, si in itertools.product(range(r), range(r)):
            hh, ww = p0 * st - pad + ri, q0 * st - pad + si
            if 0 <= hh < h and 0 <= ww < w:
                want_dx[n0, :, hh, ww] = Wk[k0, :, ri, si]
                want_dw[k0, :, ri, si] = X[n0, :, hh, ww]
        assert np.array_equal(DX.view(np.uint16), want_dx.view(np.uint16))
        # +0 and -0 are both exact zeros of a sum with no terms
        assert np.array_equal(DW.astype(np.float64), want_dw.astype(np.float64))


@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
def test_one_by_one_is_gemm(layout):
    n, c, h, w, k = 2, 16, 5, 3, 12
    shp = oracle.conv_shape(n, c, h, w, k, 1, 1, 1, 0, layout)
    x, wt, _ = _inputs(shp, seed=5)
    y64, _ = oracle.conv_fwd(shp, x, wt)
    lay = 0 if layout == "NHWC" else 1
    X = np.moveaxis(_to_nchw(x.astype(np.float64), lay), 1, -1).reshape(-1, c)
    Wm = _filter_to_kcrs(wt.astype(np.float64), lay).reshape(k, c)
    ref = (X @ Wm.T).reshape(n, h, w, k)
    Y = np.moveaxis(_to_nchw(y64, lay), 1, -1)
    assert np.allclose(Y, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
def test_sampled_equals_full(layout):
    shp = oracle.conv_shape(2, 8, 9, 7, 6, 3, 3, 2, 1, layout)
    x, wt, dy = _inputs(shp, seed=9)
    y64, _ = oracle.conv_fwd(shp, x, wt)
    dx64, _ = oracle.conv_dgrad(shp, dy, wt)
    dw64, _ = oracle.conv_wgrad(shp, x, dy)
    rng = np.random.default_rng(0)
    for full, fn, a, b in [(y64, oracle.conv_fwd_at, x, wt), (dx64, oracle.conv_dgrad_at, dy, wt),
                           (dw64, oracle.conv_wgrad_at, x, dy)]:
        idx = rng.integers(0, full.size, 200)
        got = fn(shp, a, b, idx)
        assert np.array_equal(got, full.reshape(-1)[idx])


@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
def test_dgrad_add(layout):
    shp = oracle.conv_shape(2, 8, 9, 7, 6, 3, 3, 2, 1, layout)
    x, wt, dy = _inputs(shp, seed=13)
    addend = synth.normal_f16(x.shape, 1.0, 13, 9)
    dx64, _ = oracle.conv_dgrad(shp, dy, wt)
    a64, a16 = oracle.conv_dgrad_add(shp, dy, wt, addend)
    # the addend enters the float64 sum before the single rounding
    assert np.allclose(a64, dx64 + addend.astype(np.float64), rtol=0, atol=1e-15)
    assert np.array_equal(a16.view(np.uint16), a64.astype(np.float16).view(np.uint16))
    # with a zero gradient the result is the addend, bit for bit (-0 + 0 aside)
    z64, z16 = oracle.conv_dgrad_add(shp, np.zeros_like(dy), wt, addend)
    assert np.array_equal(z16.astype(np.float64), addend.astype(np.float64))
