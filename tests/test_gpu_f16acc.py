"""GPU parity of the strict binary16-arithmetic mode (the literal reading of
"all arithmetic in FP16", Section 5.2) against the oracle, and the size of
what the float32 accumulators of the default path buy.

- fp16_sgd_step_f16: bit-exact against the oracle's three binary16 fmas.
- Convolutions with accum = 1: every output a chain of binary16 fmas from +0
  in the declared order (forward taps row-major then channels; data
  gradient the reaching taps row-major then output channels; weight
  gradient the output pixels in order).  Each step is one IEEE rounding of
  an exact value, so the result is one bit pattern: bit-exact against the
  oracle (NaN by class), on every element for small shapes (channel and
  filter tails, strides, padding, 7x7, more than 1,024 channels) and on
  sampled outputs at the conv2_x (batch 32) and conv4_x (batch 128) 3x3
  layers.
- The study: the binary16 chain's error against the exact sums is reported
  next to the default path's (one rounding of a float32 sum)."""

import numpy as np
import pytest
import torch

import oracle
import paper_1911_07384_amd as F
from gpu_util import ConvCase, dev, host, note, require_gpu
from paper_1911_07384_amd import synth

pytestmark = pytest.mark.gpu


def _sgd_inputs(n, seed):
    w = synth.normal_f16((n,), 0.05, seed, 1)
    g = synth.normal_f16((n,), 1e-3, seed, 2)
    m = synth.normal_f16((n,), 1e-2, seed, 3)
    return w, g, m


@pytest.mark.parametrize("n", [1, 7, 8, 1000, 65541])
@pytest.mark.parametrize("lr,mom,wd", [(0.1, 0.9, 1e-4), (2.0 ** -14, 0.9, 1e-4), (0.1, 0.9, 0.0)])
def test_sgd_f16_bit_exact(n, lr, mom, wd):
    require_gpu()
    w, g, m = _sgd_inputs(n, 30 + n)
    W, G, M = dev(w), dev(g), dev(m)
    note(f"[gpu] sgd_f16 n={n} lr={lr}")
    F.fp16_sgd_step_f16(W, G, M, lr=lr, momentum=mom, weight_decay=wd)
    torch.cuda.synchronize()
    ew, em = oracle.sgd_f16(w, g, m, lr, mom, wd)
    assert np.array_equal(host(W).view(np.uint16), ew.view(np.uint16))
    assert np.array_equal(host(M).view(np.uint16), em.view(np.uint16))


def test_sgd_f16_special_values():
    require_gpu()
    vals = np.array([0.0, -0.0, 2.0 ** -24, -(2.0 ** -24), 2.0 ** -14, 65504.0, -65504.0,
                     np.inf, -np.inf, np.nan, 1.0, -1.0, 2048.0, 0.5], np.float16)
    w = np.repeat(vals, len(vals))
    g = np.tile(vals, len(vals))
    m = np.roll(g, 3)
    W, G, M = dev(w), dev(g), dev(m)
    F.fp16_sgd_step_f16(W, G, M, lr=0.1, momentum=0.9, weight_decay=1e-4)
    torch.cuda.synchronize()
    ew, em = oracle.sgd_f16(w, g, m, 0.1, 0.9, 1e-4)
    for got, want in ((host(W), ew), (host(M), em)):
        nan = np.isnan(want)
        assert np.array_equal(np.isnan(got), nan)
        assert np.array_equal(got.view(np.uint16)[~nan], want.view(np.uint16)[~nan])


# (n, c, h, w, k, r, s, stride, pad)
SHAPES = [
    (2, 64, 8, 8, 64, 3, 3, 1, 1),      # 3x3, channel counts multiples of 8
    (2, 24, 9, 7, 40, 3, 3, 1, 1),      # non-square image, 24 / 40 channels
    (2, 3, 16, 16, 16, 7, 7, 2, 3),     # the stem: 3 input channels, 7x7 stride 2
    (2, 32, 9, 9, 48, 3, 3, 2, 1),      # stride 2: taps reaching each position vary
    (4, 128, 5, 5, 96, 1, 1, 1, 0),     # 1x1
    (3, 5, 6, 6, 7, 3, 3, 1, 0),        # C and K not multiples of 8, no padding
    (1, 1040, 3, 3, 12, 1, 1, 1, 0),    # more than 1,024 input channels (two LDS rounds)
    (1, 20, 4, 4, 1032, 1, 1, 2, 0),    # more than 1,024 output channels, stride-2 1x1
]


def _bit_exact(got, want, what):
    nan = np.isnan(want.astype(np.float32))
    assert np.array_equal(np.isnan(got.astype(np.float32)), nan), what
    g, w = got.view(np.uint16)[~nan], want.view(np.uint16)[~nan]
    bad = int(np.count_nonzero(g != w))
    assert bad == 0, f"{what}: {bad} of {g.size} outputs differ"


@pytest.mark.parametrize("shape", SHAPES, ids=["n{}c{}h{}w{}k{}r{}s{}st{}p{}".format(*s) for s in SHAPES])
@pytest.mark.parametrize("which", ["fwd", "dgrad", "wgrad"])
def test_conv_f16acc_bit_exact(shape, which):
    require_gpu()
    n, c, h, w, k, r, s, st, pad = shape
    case = ConvCase(n, c, h, w, k, r, s, st, pad, seed=40, dy_std=1.0, accum=1)
    got = case.run(which)
    fn = {"fwd": lambda: oracle.conv_fwd_f16acc(case.shp, case.x, case.w),
          "dgrad": lambda: oracle.conv_dgrad_f16acc(case.shp, case.dy, case.w),
          "wgrad": lambda: oracle.conv_wgrad_f16acc(case.shp, case.x, case.dy)}[which]
    _bit_exact(got, fn(), f"{which} {case.label}")


def test_conv_f16acc_special_values():
    # subnormal products, signed zeros, overflow to inf and NaN inputs take
    # the same IEEE path on both sides
    require_gpu()
    vals = np.array([0.0, -0.0, 2.0 ** -24, -(2.0 ** -24), 2.0 ** -14, 1.0, -1.0, 65504.0, -65504.0,
                     np.inf, np.nan, 2048.0, 0.5, 3.0], np.float16)
    rng = np.random.default_rng(9)
    x = rng.choice(vals, (2, 5, 5, 8)).astype(np.float16)
    wt = rng.choice(vals, (8, 3, 3, 8)).astype(np.float16)
    dy = rng.choice(vals, (2, 5, 5, 8)).astype(np.float16)
    case = ConvCase(2, 8, 5, 5, 8, 3, 3, 1, 1, x=x, wt=wt, dy=dy, accum=1)
    _bit_exact(case.run("fwd"), oracle.conv_fwd_f16acc(case.shp, x, wt), "fwd special")
    _bit_exact(case.run("dgrad"), oracle.conv_dgrad_f16acc(case.shp, dy, wt), "dgrad special")
    _bit_exact(case.run("wgrad"), oracle.conv_wgrad_f16acc(case.shp, x, dy), "wgrad special")


def _sampled(case, which, nsamp, seed):
    size = {"fwd": np.prod(case.ys), "dgrad": np.prod(case.xs), "wgrad": np.prod(case.ws)}[which]
    idx = np.random.default_rng(seed).choice(int(size), min(nsamp, int(size)), replace=False)
    idx = np.unique(np.concatenate([idx, [0, int(size) - 1]]))
    fn = {"fwd": lambda: oracle.conv_fwd_f16acc_at(case.shp, case.x, case.w, idx),
          "dgrad": lambda: oracle.conv_dgrad_f16acc_at(case.shp, case.dy, case.w, idx),
          "wgrad": lambda: oracle.conv_wgrad_f16acc_at(case.shp, case.x, case.dy, idx)}[which]
    return idx, fn()


@pytest.mark.parametrize("which", ["fwd", "dgrad", "wgrad"])
def test_conv_f16acc_full_size_sampled(which):
    """The conv4_x 3x3 layer at batch 128 (2,304- and 25,088-term chains),
    bit-exact on 1,000 sampled outputs plus the first and the last."""
    require_gpu()
    case = ConvCase(128, 256, 14, 14, 256, 3, 3, 1, 1, seed=43, dy_std=1e-2, accum=1)
    got = case.run(which).reshape(-1)
    idx, want = _sampled(case, which, 1000, 44)
    _bit_exact(got[idx], want, f"{which} {case.label} sampled")


def test_f16acc_rejects_nchw_and_fused_forms():
    require_gpu()
    d = F.conv_desc(1, 8, 4, 4, 8, 1, 1, layout="NCHW", accum=1)
    t = torch.zeros(128, dtype=torch.float16, device="cuda")
    with pytest.raises(F.Fp16Error):
        F.fp16_conv_fwd(d, t, t, t, F.workspace(1 << 16))
    d = F.conv_desc(1, 8, 4, 4, 8, 1, 1, accum=1)
    a, b = torch.zeros(128, dtype=torch.float16, device="cuda"), torch.zeros(128, dtype=torch.float16, device="cuda")
    with pytest.raises(F.Fp16Error) as e:
        F.fp16_conv_dgrad_add(d, t, a, b, b.clone(), F.workspace(1 << 16))
    assert e.value.status == 7


def test_what_float32_accumulators_buy(capsys):
    """Relative RMS error against the exact sums, default vs binary16
    chains, on a 3x3 layer with reductions of 1152 (fwd, dgrad) and 392
    (wgrad) terms; the binary16 chains must be clearly worse."""
    require_gpu()
    rows = []
    for accum in (0, 1):
        case = ConvCase(2, 128, 14, 14, 128, 3, 3, 1, 1, seed=41, dy_std=1.0, accum=accum)
        for which in ("fwd", "dgrad", "wgrad"):
            got = case.run(which).astype(np.float64)
            ref64 = case.oracle(which)[0]
            rel = float(np.sqrt(np.mean((got - ref64) ** 2)) / np.sqrt(np.mean(ref64 ** 2)))
            rows.append((accum, which, rel))
    with capsys.disabled():
        for accum, which, rel in rows:
            print(f"\n[f16acc study] accum={accum} {which}: relative RMS error {rel:.3e}", end="")
        print()
    err = {(a, w): e for a, w, e in rows}
    for which in ("fwd", "dgrad", "wgrad"):
        assert err[(1, which)] > 3 * err[(0, which)]


def test_long_reduction_stagnates_in_binary16(capsys):
    """The conv2_x 3x3 weight gradient at batch 32: each output chains
    100,352 products.  On 2,000 sampled outputs the binary16 chain is
    bit-exact against the oracle's and, against the exact sums, far worse
    than the default path: once the accumulator's spacing exceeds a term,
    the term is lost (stagnation, the mantissa-underflow discussion of
    Sections 2 and 4.2)."""
    require_gpu()
    idx = np.random.default_rng(3).choice(64 * 3 * 3 * 64, 2000, replace=False)
    rows = {}
    for accum in (0, 1):
        case = ConvCase(32, 64, 56, 56, 64, 3, 3, 1, 1, seed=42, dy_std=1e-2, accum=accum)
        got = case.run("wgrad").reshape(-1)[idx]
        ref = case.oracle_at("wgrad", idx)
        if accum:
            _bit_exact(got, oracle.conv_wgrad_f16acc_at(case.shp, case.x, case.dy, idx),
                       "conv2_x wgrad N=32 binary16 chains")
        g = got.astype(np.float64)
        rows[accum] = float(np.sqrt(np.mean((g - ref) ** 2)) / np.sqrt(np.mean(ref ** 2)))
    with capsys.disabled():
        print(f"\n[f16acc study] wgrad, 100352-term reductions: relative RMS error "
              f"default {rows[0]:.3e}, binary16 chains {rows[1]:.3e}")
    assert rows[0] < 1e-3
    assert rows[1] > 10 * rows[0]
