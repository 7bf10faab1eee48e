"""GPU parity of the strict binary16-arithmetic mode (the literal reading of
"all arithmetic in FP16", Section 5.2) against the oracle, and the size of
what the float32 accumulators of the default path buy.

- fp16_sgd_step_f16: bit-exact against the oracle's three binary16 fmas.
- Convolutions with accum = 1 (binary16 accumulator rounded after every 16
  terms): the oracle sums each block of 16 in float64, the matrix core in
  float32, so a block's rounding can differ where the running sum lies
  within float32 rounding of a binary16 rounding boundary; the difference,
  one ulp of the running sum, is then carried, and cancellation later in the
  reduction can make it many ulps of a small final value.  The running sums
  are of the order of the outputs' RMS, so the bar is: >= 99% of outputs
  bit-identical and every output within 4 binary16 ulps of
  max(|oracle value|, RMS of the oracle outputs).
- The study: on a 3x3 layer the binary16 accumulator's error against the
  exact sums is reported next to the default path's (one rounding)."""

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
    (2, 64, 8, 8, 64, 3, 3, 1, 1),     # several k-blocks per tap
    (2, 24, 9, 7, 40, 3, 3, 1, 1),     # channels not multiples of 16: blocks straddle taps
    (2, 3, 16, 16, 16, 7, 7, 2, 3),    # the stem: 3 channels padded to 8
    (2, 32, 9, 9, 48, 3, 3, 2, 1),     # stride 2: data-gradient phases
    (4, 128, 5, 5, 96, 1, 1, 1, 0),    # 1x1
]


def _ulp16(m):
    """binary16 ulp at magnitude m (the subnormal quantum below 2^-14)."""
    m = np.maximum(np.abs(m), 2.0 ** -14)
    return 2.0 ** (np.floor(np.log2(m)) - 10)


def _close(got, want, what):
    g, w = got.astype(np.float64), want.astype(np.float64)
    assert np.all(np.isfinite(g)), what
    frac_exact = float(np.mean(got.view(np.uint16) == want.view(np.uint16)))
    scale = _ulp16(np.maximum(np.abs(w), np.sqrt(np.mean(w ** 2))))
    worst = float(np.max(np.abs(g - w) / scale))
    assert frac_exact >= 0.99 and worst <= 4, f"{what}: exact {frac_exact:.4f}, worst {worst:.2f} ulp"
    return frac_exact, worst


@pytest.mark.parametrize("shape", SHAPES, ids=["n{}c{}h{}w{}k{}r{}s{}st{}p{}".format(*s) for s in SHAPES])
@pytest.mark.parametrize("which", ["fwd", "dgrad", "wgrad"])
def test_conv_f16acc_parity(shape, which):
    require_gpu()
    n, c, h, w, k, r, s, st, pad = shape
    case = ConvCase(n, c, h, w, k, r, s, st, pad, seed=40, dy_std=1.0, accum=1)
    got = case.run(which)
    fn = {"fwd": lambda: oracle.conv_fwd_f16acc(case.shp, case.x, case.w),
          "dgrad": lambda: oracle.conv_dgrad_f16acc(case.shp, case.dy, case.w),
          "wgrad": lambda: oracle.conv_wgrad_f16acc(case.shp, case.x, case.dy)}[which]
    _close(got, fn(), f"{which} {case.label}")


def test_f16acc_rejects_nchw():
    require_gpu()
    d = F.conv_desc(1, 8, 4, 4, 8, 1, 1, layout="NCHW", accum=1)
    t = torch.zeros(128, dtype=torch.float16, device="cuda")
    with pytest.raises(F.Fp16Error):
        F.fp16_conv_fwd(d, t, t, t, F.workspace(1 << 16))


def test_what_float32_accumulators_buy(capsys):
    """Relative RMS error against the exact sums, default vs binary16
    accumulation, on a 3x3 layer with reductions of 1152 (fwd, dgrad) and
    392 (wgrad) terms; the binary16 accumulator must be clearly worse."""
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
    """The conv2_x 3x3 weight gradient at batch 32: each output sums 100,352
    products.  Against the exact sums (2,000 sampled outputs), the default
    path keeps one rounding's error; the binary16 accumulator loses the
    small block contributions once its ulp exceeds them (stagnation,
    Section 2's mantissa-underflow discussion) and is far worse."""
    require_gpu()
    idx = np.random.default_rng(3).choice(64 * 3 * 3 * 64, 2000, replace=False)
    rows = {}
    for accum in (0, 1):
        case = ConvCase(32, 64, 56, 56, 64, 3, 3, 1, 1, seed=42, dy_std=1e-2, accum=accum)
        got = case.run("wgrad").reshape(-1)[idx].astype(np.float64)
        ref = case.oracle_at("wgrad", idx)
        rows[accum] = float(np.sqrt(np.mean((got - ref) ** 2)) / np.sqrt(np.mean(ref ** 2)))
    with capsys.disabled():
        print(f"\n[f16acc study] wgrad, 100352-term reductions: relative RMS error "
              f"default {rows[0]:.3e}, binary16 accumulation {rows[1]:.3e}")
    assert rows[0] < 1e-3
    assert rows[1] > 10 * rows[0]
