"""Gradual underflow through the convolution passes (IEEE subnormals, no flush
to zero; Section 4.1 names the underflow risk, Section 4.2 the mantissa
underflow of small updates).

Workload: the conv4_x 3x3 256->256 layer at 14x14 and batch 128, with output
gradients of log-uniform magnitude in [2^-24, 2^-10] and random sign: most of
them are binary16 subnormals.  Flushing subnormal operands anywhere (matrix
core inputs, conversions, stores) would move the weight gradient by several
percent of its RMS and fail the 1e-2 bar.  The SGD side of the same stress
(updates in the subnormal range) is in test_gpu_sgd.py."""

import numpy as np
import pytest

from gpu_util import ConvCase, require_gpu
from paper_1911_07384_amd import synth

pytestmark = pytest.mark.gpu


def _case(x_scale=1.0, n=128):
    c = ConvCase(n, 256, 14, 14, 256, 3, 3, 1, 1, "NHWC", seed=5)
    c.dy = synth.loguniform_f16(c.ys, -24.0, -10.0, 5, 3)
    if x_scale != 1.0:
        c.x = (c.x.astype(np.float64) * x_scale).astype(np.float16)
    return c


def _sampled(case, which, got, k=3000):
    rng = np.random.default_rng(11)
    flat = got.reshape(-1)
    idx = np.unique(rng.integers(0, flat.size, k))
    ref = case.oracle_at(which, idx)
    g = flat[idx].astype(np.float64)
    rms = np.sqrt(np.mean(ref ** 2))
    return g, ref, rms


def test_inputs_are_mostly_subnormal():
    c = _case(n=2)
    a = np.abs(c.dy.astype(np.float64))
    assert np.mean((a < 2.0 ** -14) & (a > 0)) > 0.6


@pytest.mark.parametrize("which", ["wgrad", "dgrad"])
def test_subnormal_gradients(which):
    require_gpu()
    c = _case()
    got = c.run(which)
    g, ref, rms = _sampled(c, which, got)
    assert np.max(np.abs(g - ref)) <= 1e-2 * rms, (np.max(np.abs(g - ref)), rms)
    if which == "dgrad":
        # the data gradient itself lands largely in the subnormal range
        a = np.abs(got.astype(np.float64))
        assert np.mean((a > 0) & (a < 2.0 ** -14)) > 0.05


def test_subnormal_weight_gradient_outputs():
    # x scaled by 2^-10: the weight gradient itself is mostly subnormal
    require_gpu()
    c = _case(x_scale=2.0 ** -10)
    got = c.run("wgrad")
    g, ref, rms = _sampled(c, "wgrad", got)
    a = np.abs(ref)
    assert np.mean((a > 0) & (a < 2.0 ** -14)) > 0.5
    # bar: 1e-2 * RMS, or one subnormal quantum (2^-24) where the values are that small
    assert np.all(np.abs(g - ref) <= np.maximum(1e-2 * rms, 2.0 ** -24)), np.max(np.abs(g - ref))
