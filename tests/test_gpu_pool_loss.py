"""GPU parity of the pooling layers and the classifier loss (the parts of
ResNet-50 around the residual blocks, Section 5.1) against the oracle.

Max pooling outputs, tap indices and gradients, and both average-pooling
directions are bit-exact (selections and exact float64 sums, one rounding).
The loss gradient and bias gradient are float64 computations rounded once to
binary16 on both sides; they may differ only where the two float64 values
straddle a rounding boundary, so the bar is at most 1 ulp anywhere and
bit-exact on all but a handful of entries."""

import numpy as np
import pytest
import torch

import oracle
import paper_1911_07384_amd as F
from gpu_util import dev, host, note, require_gpu, ulp_dist
from paper_1911_07384_amd import synth

pytestmark = pytest.mark.gpu


def _maxpool_input(shape, seed, special=False):
    x = synth.normal_f16(shape, 1.0, seed, 1)
    # half-integer grid: many exact ties inside windows
    x = (np.round(x.astype(np.float64) * 2) / 2).astype(np.float16)
    if special:
        flat = x.reshape(-1)
        rng = np.random.default_rng(seed)
        pos = rng.choice(flat.size, max(4, flat.size // 500), replace=False)
        vals = np.array([np.nan, -0.0, np.inf, -np.inf, 65504, 2.0 ** -24], np.float16)
        flat[pos] = vals[np.arange(pos.size) % vals.size]
    return x


MAXPOOL = [  # n, c, h, w, r, stride, pad, layout, special
    (2, 64, 112, 112, 3, 2, 1, "NHWC", True),   # the ResNet-50 stem pool, batch 2
    (3, 16, 17, 13, 3, 2, 1, "NHWC", True),     # ragged sizes
    (2, 8, 8, 10, 3, 2, 1, "NHWC", True),       # even sizes: the last block's second windows are past the edge
    (2, 3, 9, 10, 3, 2, 1, "NHWC", True),       # C not a multiple of 8
    (2, 5, 11, 9, 3, 2, 1, "NCHW", True),
    (1, 8, 6, 6, 2, 2, 0, "NHWC", False),
    (1, 8, 7, 7, 3, 1, 1, "NHWC", False),       # overlapping stride-1 windows
    (1, 8, 4, 4, 3, 3, 2, "NHWC", False),       # windows overhanging both edges
]


@pytest.mark.parametrize("case", MAXPOOL)
def test_maxpool_fwd_bwd_bit_exact(case):
    require_gpu()
    n, c, h, w, r, st, pad, layout, special = case
    xs = (n, h, w, c) if layout == "NHWC" else (n, c, h, w)
    x = _maxpool_input(xs, 11 + h, special)
    shp = oracle.pool_shape(n, c, h, w, r, r, st, pad, layout)
    d = F.pool_desc(n, c, h, w, r, r, st, pad, layout)
    P, Q = F.fp16_pool_out_dims(d)
    assert (P, Q) == oracle.pool_out_dims(shp)
    ys = (n, P, Q, c) if layout == "NHWC" else (n, c, P, Q)
    dy = synth.normal_f16(ys, 1e-2, 11 + h, 2)
    y_ref, idx_ref = oracle.maxpool_fwd(shp, x)
    dx_ref = oracle.maxpool_bwd(shp, x, dy)
    note(f"[gpu] maxpool {case}")
    xd = dev(x)
    y = torch.empty(ys, dtype=torch.float16, device="cuda")
    idx = torch.empty(ys, dtype=torch.uint8, device="cuda")
    F.fp16_maxpool_fwd(d, xd, y, idx)
    dx = torch.full(xs, float("nan"), dtype=torch.float16, device="cuda")
    F.fp16_maxpool_bwd(d, idx, dev(dy), dx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(y).view(np.uint16), y_ref.view(np.uint16))
    np.testing.assert_array_equal(host(idx), idx_ref)
    np.testing.assert_array_equal(host(dx).view(np.uint16), dx_ref.view(np.uint16))


def test_maxpool_full_resnet50_stem_pool():
    # batch 128, [128, 112, 112, 64] -> [128, 56, 56, 64], the size the training step runs
    require_gpu()
    n, c, h = 128, 64, 112
    shp = oracle.pool_shape(n, c, h, h, 3, 3, 2, 1, "NHWC")
    d = F.pool_desc(n, c, h, h, 3, 3, 2, 1, "NHWC")
    x = synth.normal_f16((n, h, h, c), 1.0, 21, 1)
    dy = synth.normal_f16((n, 56, 56, c), 1e-3, 21, 2)
    y_ref, idx_ref = oracle.maxpool_fwd(shp, x)
    dx_ref = oracle.maxpool_bwd(shp, x, dy)
    note("[gpu] maxpool full 128x112x112x64")
    y = torch.empty((n, 56, 56, c), dtype=torch.float16, device="cuda")
    idx = torch.empty((n, 56, 56, c), dtype=torch.uint8, device="cuda")
    F.fp16_maxpool_fwd(d, dev(x), y, idx)
    dx = torch.empty((n, h, h, c), dtype=torch.float16, device="cuda")
    F.fp16_maxpool_bwd(d, idx, dev(dy), dx)
    torch.cuda.synchronize()
    assert np.array_equal(host(y).view(np.uint16), y_ref.view(np.uint16))
    assert np.array_equal(host(idx), idx_ref)
    assert np.array_equal(host(dx).view(np.uint16), dx_ref.view(np.uint16))


AVG = [  # n, c, h, w, layout
    (128, 2048, 7, 7, "NHWC"),   # ResNet-50's pool at batch 128
    (3, 24, 5, 6, "NHWC"),
    (2, 5, 7, 7, "NHWC"),        # C not a multiple of 8
    (2, 6, 4, 3, "NCHW"),
    (4, 8, 1, 1, "NHWC"),        # a 1x1 grid
]


@pytest.mark.parametrize("case", AVG)
def test_avgpool_fwd_bwd_bit_exact(case):
    require_gpu()
    n, c, h, w, layout = case
    xs = (n, h, w, c) if layout == "NHWC" else (n, c, h, w)
    x = synth.normal_f16(xs, 1.0, 31 + c, 1)
    x.reshape(-1)[:3] = np.array([-0.0, 65504, 2.0 ** -24], np.float16)
    dy = synth.normal_f16((n, c), 1e-3, 31 + c, 2)
    dy.reshape(-1)[:2] = np.array([2.0 ** -24, -0.0], np.float16)
    shp = oracle.pool_shape(n, c, h, w, h, w, 1, 0, layout)
    d = F.pool_desc(n, c, h, w, h, w, 1, 0, layout)
    _, y_ref = oracle.avgpool_fwd(shp, x)
    dx_ref = oracle.avgpool_bwd(shp, dy)
    note(f"[gpu] avgpool {case}")
    y = torch.empty((n, c), dtype=torch.float16, device="cuda")
    F.fp16_avgpool_fwd(d, dev(x), y)
    dx = torch.empty(xs, dtype=torch.float16, device="cuda")
    F.fp16_avgpool_bwd(d, dev(dy), dx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(y).view(np.uint16), y_ref.view(np.uint16))
    np.testing.assert_array_equal(host(dx).view(np.uint16), dx_ref.view(np.uint16))


LOSS = [  # n, k, z_std, bias_std
    (128, 1000, 1.0, 0.1),   # ResNet-50's classifier at batch 128
    (128, 1000, 0.01, 0.0),  # near-uniform: gradients in the subnormal range
    (3, 37, 8.0, 1.0),       # K not a multiple of anything, large spread
    (1, 1, 1.0, 1.0),        # degenerate: one class, zero loss and gradient
    (5, 300, 2000.0, 0.0),   # large logits: the max shift keeps exp finite
]


@pytest.mark.parametrize("case", LOSS)
def test_softmax_ce_parity(case):
    require_gpu()
    n, k, zs, bs = case
    z = synth.normal_f16((n, k), zs, 41 + k, 1)
    b = synth.normal_f16((k,), bs, 41 + k, 2) if bs else np.zeros(k, np.float16)
    lab = synth.labels(n, k, 41 + k, 3)
    ref = oracle.softmax_ce(z, b, lab)
    note(f"[gpu] softmax_ce {case}")
    loss = torch.empty(n, dtype=torch.float32, device="cuda")
    dz = torch.empty((n, k), dtype=torch.float16, device="cuda")
    db = torch.empty(k, dtype=torch.float16, device="cuda")
    F.fp16_softmax_ce(n, k, dev(z), dev(b), torch.from_numpy(lab).to("cuda"), loss, dz, db)
    torch.cuda.synchronize()
    got = host(loss).astype(np.float64)
    np.testing.assert_allclose(got, ref["loss_rows"], rtol=2 ** -23, atol=1e-30)
    du = ulp_dist(host(dz), ref["dz"])
    assert du.max() <= 1 and np.count_nonzero(du) <= max(2, du.size // 10000), du.max()
    bu = ulp_dist(host(db), ref["db"])
    assert bu.max() <= 1


def test_softmax_ce_in_place():
    # dz may equal z: same results as out of place
    require_gpu()
    n, k = 16, 100
    z = synth.normal_f16((n, k), 1.0, 51, 1)
    b = synth.normal_f16((k,), 0.1, 51, 2)
    lab = torch.from_numpy(synth.labels(n, k, 51, 3)).to("cuda")
    loss = torch.empty(n, dtype=torch.float32, device="cuda")
    db = torch.empty(k, dtype=torch.float16, device="cuda")
    out = torch.empty((n, k), dtype=torch.float16, device="cuda")
    F.fp16_softmax_ce(n, k, dev(z), dev(b), lab, loss, out, db)
    zz = dev(z)
    F.fp16_softmax_ce(n, k, zz, dev(b), lab, loss, zz, db)
    torch.cuda.synchronize()
    assert torch.equal(zz.view(torch.int16), out.view(torch.int16))


# (n, c, h, w, stride, pad, use_stats, special): BN + ReLU fused into a 3x3 max
# pool; "special" puts NaN, infinities and ties into x under given statistics
BN_POOL = [
    (2, 64, 112, 112, 2, 1, False, False),   # the ResNet-50 stem's BN + pool at N = 2
    (32, 64, 112, 112, 2, 1, False, False),  # ... at batch 32
    (3, 8, 7, 9, 2, 1, False, False),        # one chunk per pixel, odd sides, ragged windows
    (2, 16, 10, 6, 1, 1, False, False),      # stride 1
    (2, 128, 9, 11, 2, 0, True, False),      # no padding, given statistics
    (2, 256, 5, 5, 3, 2, True, True),        # stride 3, pad 2; NaN, infinities and ties
    (2, 256, 20, 64, 2, 1, False, False),    # 32 channel chunks per pixel
    (2, 256, 9, 7, 2, 1, True, True),        # the stride-2 column strips: NaN, infinities, ties
    (2, 64, 35, 21, 2, 1, False, False),     # ragged last row strip (18 rows) and column strip
]


@pytest.mark.parametrize("case", BN_POOL, ids=[str(c) for c in BN_POOL])
def test_bn_relu_maxpool_matches_the_two_calls(case):
    require_gpu()
    n, c, h, w, st, pad, given, special = case
    bd = F.bn_desc(n, c, h, w, "NHWC", 1e-5, 1.0, True)
    pd = F.pool_desc(n, c, h, w, 3, 3, st, pad)
    p, q = F.fp16_pool_out_dims(pd)
    x = synth.normal_f16((n, h, w, c), 1.0, 60 + c, 1, mean=0.3)
    gamma = synth.normal_f16((c,), 0.3, 60 + c, 2, mean=1.0)
    beta = synth.normal_f16((c,), 0.3, 60 + c, 3)
    G, B = dev(gamma), dev(beta)
    ws = F.workspace(F.fp16_bn_workspace_bytes(bd))
    S = torch.empty(2 * c, dtype=torch.float32, device="cuda")
    Z = torch.empty((n, h, w, c), dtype=torch.float16, device="cuda")
    note(f"[gpu] bn statistics {case}")
    F.fp16_bn_relu(bd, dev(x), G, B, None, Z, S, ws)
    if special:
        x = x.copy()
        flat = x.reshape(-1)
        flat[::2] = flat[1::2]  # equal neighbours: ties inside windows
        flat[::97] = np.float16(np.nan)
        flat[5::89] = np.float16(np.inf)
        flat[7::83] = np.float16(-np.inf)
    X = dev(x)
    if given:
        bd = F.bn_desc(n, c, h, w, "NHWC", 1e-5, 1.0, True, use_stats=True)
    Y0 = torch.empty((n, p, q, c), dtype=torch.float16, device="cuda")
    I0 = torch.empty((n, p, q, c), dtype=torch.uint8, device="cuda")
    S0 = S.clone()
    note(f"[gpu] bn + maxpool (two calls) {case}")
    F.fp16_bn_relu(bd, X, G, B, None, Z, S0, ws)
    F.fp16_maxpool_fwd(pd, Z, Y0, I0)
    S1 = S.clone() if given else torch.full_like(S, float("nan"))
    Y1 = torch.full_like(Y0, float("nan"))
    I1 = torch.full_like(I0, 0xEE)
    note(f"[gpu] bn_relu_maxpool {case}")
    F.fp16_bn_relu_maxpool(bd, pd, X, G, B, S1, Y1, I1, ws)
    torch.cuda.synchronize()
    assert np.array_equal(host(S1), host(S0))
    assert np.array_equal(host(Y1).view(np.uint16), host(Y0).view(np.uint16))
    assert np.array_equal(host(I1), host(I0))
    if n * c * h * w <= 1 << 21:
        # and against the oracle: the declared apply with these statistics, pooled
        s = host(S0)
        z = oracle.bn_apply_f32(oracle.bn_shape(n, c, h, w), x, gamma, beta, s[:c], s[c:], None,
                                1.0, True)
        y, idx = oracle.maxpool_fwd(oracle.pool_shape(n, c, h, w, 3, 3, st, pad), z)
        assert np.array_equal(host(Y1).view(np.uint16), y.view(np.uint16))
        assert np.array_equal(host(I1), idx)
