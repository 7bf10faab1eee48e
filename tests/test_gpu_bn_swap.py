"""GPU parity of the BN swap (Section 4.1: the shortcut joins before gamma in
a residual block's last BN) in fp16_bn_relu / fp16_bn_relu_bwd, against the
oracle.

Bars as for the ordinary BN (test_gpu_bn.py): forward with its own
statistics within 1 ulp, with given statistics bit-exact against the
declared float32 swap sequence; backward dx within 1e-2 * RMS, dgamma (now
S2 + S3) and dbeta within 1 ulp or 1e-2 * RMS.  The shortcut gradient
gamma * s * dy is bit-exact when s is a power of two (the float32 product of
binary16 values is then exact before its one rounding), else within 1 ulp."""

import numpy as np
import pytest

import oracle
import paper_1911_07384_amd as F
from gpu_util import require_gpu, ulp_dist
from test_gpu_bn import EPS, _bwd_gpu, _fwd_gpu, _inputs

pytestmark = pytest.mark.gpu

# (n, c, h, w, layout, post_scale, relu)
CASES = [
    (2, 256, 7, 7, "NHWC", 0.25, True),
    (3, 2048, 2, 3, "NHWC", 0.25, True),    # widest vector case
    (2, 64, 9, 7, "NHWC", 0.25, True),
    (2, 16, 5, 5, "NHWC", 0.25, False),     # no ReLU
    (2, 24, 5, 3, "NHWC", 0.25, True),      # generic path
    (2, 32, 6, 5, "NCHW", 0.25, True),      # NCHW
    (2, 64, 9, 7, "NHWC", 0.3, True),       # a multiplier that is not a power of two
    (32, 256, 56, 56, "NHWC", 0.25, True),  # the conv2_x block-last BN at batch 32
]


def _ids(c):
    return "n{}c{}h{}w{}{}s{}{}".format(c[0], c[1], c[2], c[3], c[4], c[5], "relu" if c[6] else "")


@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_swap_forward(case):
    n, c, h, w, lay, s, relu = case
    shp = oracle.bn_shape(n, c, h, w, lay)
    _, x, gamma, beta, res, _ = _inputs(n, c, h, w, lay, 10)
    ref = oracle.bn_fwd(shp, x, gamma, beta, res, EPS, s, relu, swap=True)
    y, st = _fwd_gpu(F.bn_desc(n, c, h, w, lay, EPS, s, relu, swap=True), x, gamma, beta, res)
    d = ulp_dist(y, ref["y"])
    absd = np.abs(y.astype(np.float64) - ref["y"].astype(np.float64))
    bound = 2.0 ** -22 * (1 + np.abs(s * beta.astype(np.float64)).max()
                          + np.abs(s * gamma.astype(np.float64)).max() * np.abs(res.astype(np.float64)))
    assert np.all((d <= 1) | (absd <= bound))
    # given statistics: bit-exact against the declared float32 swap sequence
    mean, rstd = st[:c].copy(), st[c:].copy()
    want = oracle.bn_apply_f32(shp, x, gamma, beta, mean, rstd, res, s, relu, swap=True)
    y2, _ = _fwd_gpu(F.bn_desc(n, c, h, w, lay, EPS, s, relu, use_stats=True, swap=True), x,
                     gamma, beta, res, np.concatenate([mean, rstd]))
    assert np.array_equal(y2.view(np.uint16), want.view(np.uint16))
    assert np.array_equal(y.view(np.uint16), want.view(np.uint16))


@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_swap_backward(case):
    n, c, h, w, lay, s, relu = case
    shp = oracle.bn_shape(n, c, h, w, lay)
    _, x, gamma, beta, res, dy = _inputs(n, c, h, w, lay, 11)
    st = oracle.bn_fwd(shp, x, gamma, beta, res, EPS, s, relu, swap=True)
    mean = st["mean"].astype(np.float32)
    rstd = (1.0 / np.sqrt(st["var"] + float(np.float32(EPS)))).astype(np.float32)
    stats = np.concatenate([mean, rstd])
    y = oracle.bn_apply_f32(shp, x, gamma, beta, mean, rstd, res, s, relu, swap=True)
    ref = oracle.bn_bwd(shp, x, y, dy, gamma, EPS, s, relu, want_dres=True, swap=True,
                        residual=res)
    desc = F.bn_desc(n, c, h, w, lay, EPS, s, relu, swap=True)
    dx, dg, db, dr = _bwd_gpu(desc, x, y, dy, gamma, beta, res, stats, True)
    rms = np.sqrt(np.mean(ref["dx64"] ** 2))
    assert np.max(np.abs(dx.astype(np.float64) - ref["dx64"])) <= 1e-2 * rms
    for got, r64, r16 in [(dg, ref["dgamma64"], ref["dgamma"]), (db, ref["dbeta64"], ref["dbeta"])]:
        rmsg = np.sqrt(np.mean(r64 ** 2))
        ok = (ulp_dist(got, r16) <= 1) | (np.abs(got.astype(np.float64) - r64) <= 1e-2 * rmsg)
        assert np.all(ok)
    if s in (0.25, 0.5, 1.0):
        assert np.array_equal(dr.view(np.uint16), ref["dres"].view(np.uint16))
    else:
        assert ulp_dist(dr, ref["dres"]).max() <= 1
    # mask recomputed from x, the residual and the statistics: same bits
    dx2, dg2, db2, dr2 = _bwd_gpu(desc, x, None, dy, gamma, beta, res, stats, True)
    assert np.array_equal(dx2.view(np.uint16), dx.view(np.uint16))
    assert np.array_equal(dg2.view(np.uint16), dg.view(np.uint16))
    assert np.array_equal(dr2.view(np.uint16), dr.view(np.uint16))


def test_swap_needs_the_residual():
    require_gpu()
    import torch
    d = F.bn_desc(2, 8, 4, 4, "NHWC", EPS, 0.25, True, swap=True)
    t = torch.zeros((2, 4, 4, 8), dtype=torch.float16, device="cuda")
    g = torch.ones(8, dtype=torch.float16, device="cuda")
    st = torch.zeros(16, dtype=torch.float32, device="cuda")
    ws = F.workspace(F.fp16_bn_workspace_bytes(d))
    with pytest.raises(F.Fp16Error):
        F.fp16_bn_relu(d, t, g, g, None, t, st, ws)
