"""GPU checks of the kept ReLU mask (fp16_bn_relu_m, fp16_conv_bn_relu_fwd_m,
fp16_bn_relu_bwd_m): the BN of Eq. 1-2 (Section 4.1) followed by the ReLU,
with the mask [y > 0] written by the forward and read by the backward.

Bars: every output of the _m calls bit-identical to the call without the
mask; the mask bit-exact against [y > 0] of the returned y, packed one byte
per 8 channels of a pixel, bit e for channel 8j+e."""

import numpy as np
import pytest
import torch

import paper_1911_07384_amd as F
from paper_1911_07384_amd import synth
from gpu_util import dev, host, note, require_gpu

pytestmark = pytest.mark.gpu

EPS = 1e-5

# (n, c, h, w, residual, use_stats)
CASES = [
    (2, 256, 7, 7, True, False),     # block-last BN with the shortcut
    (2, 64, 14, 14, False, False),   # no shortcut
    (3, 2048, 2, 3, True, False),    # widest vector case
    (2, 8, 5, 3, True, False),       # one byte per pixel, ragged pixel count
    (2, 256, 7, 7, True, True),      # given statistics
    (32, 256, 56, 56, True, False),  # conv2_x block-last BN at batch 32 (full size)
    (16, 2048, 7, 7, True, False),   # conv5_x block-last BN, block-major partials
]


def _ids(c):
    return "n{}c{}h{}w{}{}{}".format(c[0], c[1], c[2], c[3], "r" if c[4] else "",
                                     "given" if c[5] else "")


def _packed(y):
    """[y > 0] packed per 8 channels of a pixel, bit e = channel 8j+e."""
    pos = (y.astype(np.float32) > 0).reshape(-1, y.shape[-1] // 8, 8)
    return np.packbits(pos, axis=-1, bitorder="little").reshape(-1)


def _inputs(n, c, h, w, seed):
    xs = (n, h, w, c)
    x = synth.normal_f16(xs, 1.0, seed, 1, mean=0.2)
    gamma = synth.normal_f16((c,), 0.3, seed, 2, mean=1.0)
    beta = synth.normal_f16((c,), 0.3, seed, 3)
    res = synth.normal_f16(xs, 1.0, seed, 4)
    dy = synth.normal_f16(xs, 1e-3, seed, 5)
    return x, gamma, beta, res, dy


@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_mask_forward_and_backward(case):
    require_gpu()
    n, c, h, w, with_r, given = case
    x, gamma, beta, res, dy = _inputs(n, c, h, w, 70 + c)
    X, G, B, DY = dev(x), dev(gamma), dev(beta), dev(dy)
    R = dev(res) if with_r else None
    desc = F.bn_desc(n, c, h, w, "NHWC", EPS, 0.25, True)
    mb = F.fp16_bn_mask_bytes(desc)
    assert mb == n * h * w * c // 8
    ws = F.workspace(F.fp16_bn_workspace_bytes(desc))
    S = torch.empty(2 * c, dtype=torch.float32, device="cuda")
    Y = torch.empty_like(X)
    note(f"[gpu] bn fwd (reference) {case}")
    F.fp16_bn_relu(desc, X, G, B, R, Y, S, ws)
    if given:
        desc = F.bn_desc(n, c, h, w, "NHWC", EPS, 0.25, True, use_stats=True)
    S2 = S.clone()
    Y2 = torch.full_like(X, float("nan"))
    M = torch.full((mb,), 0xA5, dtype=torch.uint8, device="cuda")
    note(f"[gpu] bn fwd_m {case}")
    F.fp16_bn_relu_m(desc, X, G, B, R, Y2, S2, M, ws)
    torch.cuda.synchronize()
    y = host(Y)
    assert np.array_equal(host(Y2).view(np.uint16), y.view(np.uint16))
    assert np.array_equal(host(S2), host(S))
    assert np.array_equal(host(M), _packed(y))

    outs = []
    for kept in (False, True):
        DX = torch.empty_like(X)
        DG = torch.empty_like(G)
        DB = torch.empty_like(B)
        DR = torch.empty_like(X) if with_r else None
        note(f"[gpu] bn bwd{'_m' if kept else ''} {case}")
        if kept:
            F.fp16_bn_relu_bwd_m(desc, X, M, DY, G, B, S, DX, DG, DB, DR, ws)
        else:
            F.fp16_bn_relu_bwd(desc, X, None, DY, G, B, R, S, DX, DG, DB, DR, ws)
        torch.cuda.synchronize()
        outs.append([host(t).view(np.uint16) for t in (DX, DG, DB) + ((DR,) if with_r else ())])
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


# n, c, h, k, r, stride, pad, residual
CONV_CASES = [
    (2, 64, 28, 256, 1, 1, 0, True),     # block conv3 + bn3 with the shortcut (pointwise kernel)
    (4, 64, 56, 64, 3, 1, 1, False),     # 3x3 64-channel kernel, then the statistics pass
    (2, 128, 28, 128, 3, 1, 1, False),   # statistics in the convolution's epilogue
    (2, 3, 32, 64, 7, 2, 3, False),      # the stem
    (32, 64, 56, 256, 1, 1, 0, True),    # conv2_x block conv3 + bn3 at batch 32
]


@pytest.mark.parametrize("case", CONV_CASES, ids=[str(c) for c in CONV_CASES])
def test_conv_bn_mask(case):
    require_gpu()
    n, c, h, k, r, st, pad, with_res = case
    cd = F.conv_desc(n, c, h, h, k, r, r, st, pad)
    p, q = F.fp16_conv_out_dims(cd)
    bd = F.bn_desc(n, k, p, q, "NHWC", EPS, 0.25, True)
    x = synth.normal_f16((n, h, h, c), 1.0, 80 + h, 1)
    w = synth.normal_f16((k, r, r, c), synth.he_std(c * r * r), 80 + h, 2)
    gamma = synth.normal_f16((k,), 0.3, 80 + h, 3, mean=1.0)
    beta = synth.normal_f16((k,), 0.3, 80 + h, 4)
    X, W, G, B = dev(x), dev(w), dev(gamma), dev(beta)
    R = dev(synth.normal_f16((n, p, q, k), 1.0, 80 + h, 5)) if with_res else None
    ws = F.workspace(F.fp16_conv_bn_workspace_bytes(cd, bd))
    res = []
    for kept in (False, True):
        Y = torch.empty((n, p, q, k), dtype=torch.float16, device="cuda")
        Z = torch.empty_like(Y)
        S = torch.empty(2 * k, dtype=torch.float32, device="cuda")
        note(f"[gpu] conv_bn{'_m' if kept else ''} {case}")
        if kept:
            M = torch.full((F.fp16_bn_mask_bytes(bd),), 0x5A, dtype=torch.uint8, device="cuda")
            F.fp16_conv_bn_relu_fwd_m(cd, bd, X, W, G, B, R, Y, Z, S, M, ws)
        else:
            F.fp16_conv_bn_relu_fwd(cd, bd, X, W, G, B, R, Y, Z, S, ws)
        torch.cuda.synchronize()
        res.append((host(Y), host(Z), host(S)))
    (y0, z0, s0), (y1, z1, s1) = res
    assert np.array_equal(y1.view(np.uint16), y0.view(np.uint16))
    assert np.array_equal(z1.view(np.uint16), z0.view(np.uint16))
    assert np.array_equal(s1, s0)
    assert np.array_equal(host(M), _packed(z1))
