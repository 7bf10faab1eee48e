"""GPU parity of fp16_conv_bn_relu_fwd: a convolution whose epilogue also
takes the statistics of the BN that follows (ResNet-50's conv -> BN pairs,
Section 5.1; Eq. 1-2 of Section 4.1).

Bars: y bit-identical to fp16_conv_fwd; the statistics within float32
rounding of the oracle's on that y; z bit-exact against the declared float32
apply with the written statistics, and within 1 ulp of the oracle's BN."""

import numpy as np
import pytest
import torch

import oracle
import paper_1911_07384_amd as F
from gpu_util import dev, host, note, require_gpu, ulp_dist
from paper_1911_07384_amd import synth

pytestmark = pytest.mark.gpu

EPS = 1e-5

# n, c, h, k, r, stride, pad, post_scale, residual, relu, swap
CASES = [
    (2, 256, 56, 64, 1, 1, 0, 0.25, False, True, False),   # block conv1 + bn1 (register-direct kernel)
    (4, 64, 56, 64, 3, 1, 1, 0.25, False, True, False),    # 3x3 64-channel: its own kernel, then
                                                           # the BN's statistics pass
    (2, 128, 28, 128, 3, 1, 1, 0.25, False, True, False),  # 3x3 128-channel: DMA-staged kernel
                                                           # with the statistics epilogue
    (2, 64, 28, 256, 1, 1, 0, 0.25, True, True, False),    # block conv3 + bn3 with the shortcut
    (3, 64, 7, 128, 3, 1, 1, 0.25, False, True, False),    # M = 147: ragged last band
    (3, 64, 9, 64, 3, 1, 1, 0.25, False, True, False),     # M = 243, 64 channels: ragged band, narrow tile
    (2, 3, 32, 64, 7, 2, 3, 1.0, False, True, False),      # the stem, s = 1: stem kernel, then the
                                                           # BN with its own statistics pass
    (1, 3, 224, 64, 7, 2, 3, 1.0, False, True, False),     # the ResNet-50 stem at full size
    (2, 64, 14, 256, 1, 1, 0, 0.25, True, True, True),     # BN swap on the block-last BN
    (2, 128, 15, 64, 3, 2, 1, 0.25, False, False, False),  # strided, no ReLU
    (32, 256, 56, 64, 1, 1, 0, 0.25, False, True, False),  # the conv2_x block's conv1 at batch 32
    (3, 128, 9, 384, 1, 1, 0, 0.25, False, True, False),   # pointwise kernel over 128 channels,
                                                           # ragged rows and channel tiles
    (5, 64, 56, 256, 1, 1, 0, 0.25, True, True, False),    # pointwise, many tiles per workgroup
    (6, 64, 212, 64, 1, 1, 0, 0.25, False, True, False),   # 2,107 tile records (ragged): the
                                                           # statistics take the sliced two-kernel path
    (21, 64, 56, 256, 1, 1, 0, 0.25, True, True, False),   # pointwise: 515 tiles over 512 workgroup
                                                           # records, the ragged last tile in record 2
    (21, 128, 28, 512, 1, 1, 0, 0.25, True, True, False),  # pointwise over 128 channels: 129 tiles
                                                           # over 128 records (tiles 0 and 128 in one)
    (2, 64, 20, 192, 1, 1, 0, 0.25, True, False, False),  # pointwise over 64, its second pass
                                                           # applying the BN: no ReLU, ragged tile
    (3, 64, 9, 256, 1, 1, 0, 0.25, False, True, False),    # ... no shortcut, ragged rows
    (3, 256, 40, 1024, 1, 1, 0, 0.25, True, True, False),  # pointwise over 256: 38 tiles on 32 records
    (2, 256, 14, 136, 1, 1, 0, 0.25, False, True, False),  # pointwise over 256, ragged channel tile
    (4, 256, 28, 512, 1, 2, 0, 0.25, False, True, False),  # strided pointwise over 256 (the conv3_x
                                                           # shortcut's shape)
]


def _ids(c):
    return "n{}c{}h{}k{}r{}st{}{}{}{}".format(c[0], c[1], c[2], c[3], c[4], c[5],
                                             "res" if c[8] else "", "relu" if c[9] else "",
                                             "swap" if c[10] else "")


@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_conv_bn_fused(case):
    require_gpu()
    n, c, h, k, r, st, pad, s, with_res, relu, swap = case
    cd = F.conv_desc(n, c, h, h, k, r, r, st, pad)
    p, q = F.fp16_conv_out_dims(cd)
    bd = F.bn_desc(n, k, p, q, "NHWC", EPS, s, relu, swap=swap)
    x = synth.normal_f16((n, h, h, c), 1.0, 60 + h, 1)
    w = synth.normal_f16((k, r, r, c), synth.he_std(c * r * r), 60 + h, 2)
    gamma = synth.normal_f16((k,), 0.3, 60 + h, 3, mean=1.0)
    beta = synth.normal_f16((k,), 0.3, 60 + h, 4)
    res = synth.normal_f16((n, p, q, k), 1.0, 60 + h, 5) if with_res else None
    X, W, G, B = dev(x), dev(w), dev(gamma), dev(beta)
    R = dev(res) if with_res else None
    Y = torch.empty((n, p, q, k), dtype=torch.float16, device="cuda")
    Z = torch.empty_like(Y)
    S = torch.empty(2 * k, dtype=torch.float32, device="cuda")
    ws = F.workspace(F.fp16_conv_bn_workspace_bytes(cd, bd))
    note(f"[gpu] conv_bn {case}")
    F.fp16_conv_bn_relu_fwd(cd, bd, X, W, G, B, R, Y, Z, S, ws)
    Y2 = torch.empty_like(Y)
    F.fp16_conv_fwd(cd, X, W, Y2, F.workspace(F.fp16_conv_workspace_bytes(cd, F.PASS_FWD)))
    torch.cuda.synchronize()
    y, z, st_ = host(Y), host(Z), host(S)
    assert np.array_equal(y.view(np.uint16), host(Y2).view(np.uint16))
    shp = oracle.bn_shape(n, k, p, q)
    ref = oracle.bn_fwd(shp, y, gamma, beta, res, EPS, s, relu, swap=swap)
    rstd = 1.0 / np.sqrt(ref["var"] + float(np.float32(EPS)))
    assert np.allclose(st_[:k], ref["mean"], rtol=0, atol=2e-6 * (1 + np.abs(ref["mean"])).max())
    assert np.allclose(st_[k:], rstd, rtol=4e-6, atol=0)
    want = oracle.bn_apply_f32(shp, y, gamma, beta, st_[:k], st_[k:], res, s, relu, swap=swap)
    assert np.array_equal(z.view(np.uint16), want.view(np.uint16))
    assert ulp_dist(z, ref["y"]).max() <= 1


def test_conv_bn_in_place_output():
    # z may equal y: the convolution output is then replaced by the BN output
    require_gpu()
    n, c, h, k = 2, 64, 14, 64
    cd = F.conv_desc(n, c, h, h, k, 3, 3, 1, 1)
    bd = F.bn_desc(n, k, h, h, "NHWC", EPS, 0.25, True)
    x = synth.normal_f16((n, h, h, c), 1.0, 70, 1)
    w = synth.normal_f16((k, 3, 3, c), synth.he_std(c * 9), 70, 2)
    g = np.ones(k, np.float16)
    b = np.zeros(k, np.float16)
    ws = F.workspace(F.fp16_conv_bn_workspace_bytes(cd, bd))
    Y = torch.empty((n, h, h, k), dtype=torch.float16, device="cuda")
    Z = torch.empty_like(Y)
    S = torch.empty(2 * k, dtype=torch.float32, device="cuda")
    F.fp16_conv_bn_relu_fwd(cd, bd, dev(x), dev(w), dev(g), dev(b), None, Y, Z, S, ws)
    Y2 = torch.empty_like(Y)
    F.fp16_conv_bn_relu_fwd(cd, bd, dev(x), dev(w), dev(g), dev(b), None, Y2, Y2, S, ws)
    torch.cuda.synchronize()
    assert torch.equal(Y2.view(torch.int16), Z.view(torch.int16))


@pytest.mark.parametrize("alias", ["z_is_y", "z_is_residual"])
def test_conv_bn_pointwise_in_place(alias):
    # the pointwise kernel over 64 channels applies the BN in a second pass
    # that recomputes y from x: z may still be y, or the shortcut it reads
    require_gpu()
    n, c, h, k = 2, 64, 28, 256
    cd = F.conv_desc(n, c, h, h, k, 1, 1, 1, 0)
    bd = F.bn_desc(n, k, h, h, "NHWC", EPS, 0.25, True)
    x = synth.normal_f16((n, h, h, c), 1.0, 71, 1)
    w = synth.normal_f16((k, 1, 1, c), synth.he_std(c), 71, 2)
    g = synth.normal_f16((k,), 0.3, 71, 3, mean=1.0)
    b = synth.normal_f16((k,), 0.3, 71, 4)
    r = synth.normal_f16((n, h, h, k), 1.0, 71, 5)
    ws = F.workspace(F.fp16_conv_bn_workspace_bytes(cd, bd))
    Y = torch.empty((n, h, h, k), dtype=torch.float16, device="cuda")
    Z = torch.empty_like(Y)
    S = torch.empty(2 * k, dtype=torch.float32, device="cuda")
    note(f"[gpu] conv_bn pointwise in place {alias}")
    F.fp16_conv_bn_relu_fwd(cd, bd, dev(x), dev(w), dev(g), dev(b), dev(r), Y, Z, S, ws)
    Y2 = torch.empty_like(Y)
    R2 = dev(r)
    if alias == "z_is_y":
        F.fp16_conv_bn_relu_fwd(cd, bd, dev(x), dev(w), dev(g), dev(b), R2, Y2, Y2, S, ws)
        out = Y2
    else:
        F.fp16_conv_bn_relu_fwd(cd, bd, dev(x), dev(w), dev(g), dev(b), R2, Y2, R2, S, ws)
        out = R2
        assert torch.equal(Y2.view(torch.int16), Y.view(torch.int16))
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), Z.view(torch.int16))
