"""GPU checks of fp16_conv_dgrad_wf_m: the data gradient plus an addend taken
under a ReLU mask (the input gradient of a residual block, Section 4.1,
where the identity shortcut's gradient is the block-last BN's incoming
gradient through its ReLU), on every kernel the data gradient can take.

Bars: bit-identical to fp16_conv_dgrad_wf on the addend with the masked-off
elements replaced by +0 (built on the host from the mask bits), and within
the convolution bar of the oracle's data gradient plus that addend."""

import numpy as np
import pytest
import torch

import oracle
import paper_1911_07384_amd as F
from paper_1911_07384_amd import synth
from gpu_util import check_close, dev, host, note, require_gpu

pytestmark = pytest.mark.gpu

# (n, c, h, w, k, r, stride, pad): dy has k channels, dx (and the addend) c
CASES = [
    (2, 256, 14, 14, 64, 1, 1, 0),    # pointwise kernel, 64 -> 256 channels
    (3, 128, 9, 9, 64, 1, 1, 0),      # pointwise kernel, 128-channel tiles, ragged rows
    (2, 512, 7, 7, 128, 1, 1, 0),     # pointwise kernel over 128 channels
    (2, 256, 7, 7, 512, 1, 1, 0),     # DMA-staged kernel (512-long reduction)
    (2, 64, 9, 9, 512, 1, 1, 0),      # DMA-staged kernel, 64-channel tiles
    (2, 64, 10, 10, 256, 1, 1, 0),    # register-direct kernel
    (2, 64, 14, 14, 64, 3, 2, 1),     # four stride phases, register-direct
    (2, 128, 14, 14, 256, 3, 2, 1),   # four stride phases, DMA-staged
    (2, 16, 9, 9, 24, 3, 1, 1),       # LDS-staged kernel (24 channels)
    (32, 256, 56, 56, 64, 1, 1, 0),   # the conv2_x block input gradient at batch 32
    (2, 512, 14, 14, 256, 1, 1, 0),   # register-direct kernel, 256-long reduction
    (3, 1024, 40, 40, 256, 1, 1, 0),  # ... over many tiles
]


def _bits(mask, size):
    return np.unpackbits(mask, bitorder="little")[:size].astype(bool)


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
@pytest.mark.parametrize("in_place", [False, True], ids=["", "in_place"])
def test_masked_addend(case, in_place):
    require_gpu()
    n, c, h, w, k, r, st, pad = case
    if in_place and n > 3:
        pytest.skip("in place covered on the small cases")
    d = F.conv_desc(n, c, h, w, k, r, r, st, pad)
    p, q = F.fp16_conv_out_dims(d)
    seed = 90 + c + k + r
    dy = synth.normal_f16((n, p, q, k), 1e-2, seed, 1)
    wt = synth.normal_f16((k, r, r, c), synth.he_std(c * r * r), seed, 2)
    ad = synth.normal_f16((n, h, w, c), 1e-2, seed, 3)
    rng = np.random.default_rng(seed)
    mask = rng.integers(0, 256, size=n * h * w * c // 8, dtype=np.uint8)
    adm = np.where(_bits(mask, ad.size).reshape(ad.shape), ad, np.float16(0.0))
    DY, W, AD, ADM = dev(dy), dev(wt), dev(ad), dev(adm)
    M = torch.from_numpy(mask).to("cuda")
    WF = torch.empty(F.fp16_conv_dgrad_filter_bytes(d) // 2, dtype=torch.float16, device="cuda")
    ws = F.workspace(F.fp16_conv_workspace_bytes(d, F.PASS_DGRAD))
    note(f"[gpu] dgrad_wf_m {case} in_place={in_place}")
    F.fp16_conv_dgrad_filter(d, W, WF)
    ref = torch.empty_like(AD)
    F.fp16_conv_dgrad_wf(d, DY, WF, ADM, ref, ws)
    if in_place:
        DX = AD.clone()
        F.fp16_conv_dgrad_wf_m(d, DY, WF, DX, M, DX, ws)
    else:
        DX = torch.full_like(AD, float("nan"))
        F.fp16_conv_dgrad_wf_m(d, DY, WF, AD, M, DX, ws)
    torch.cuda.synchronize()
    got = host(DX)
    assert np.array_equal(got.view(np.uint16), host(ref).view(np.uint16))
    if n * h * w * c <= 1 << 20:
        shp = oracle.conv_shape(n, c, h, w, k, r, r, st, pad)
        want64, _ = oracle.conv_dgrad_add(shp, dy, wt, adm)
        check_close(got, want64, what=f"dgrad_wf_m {case}")


# (n, c, h, w, k, r, stride, pad, addend stride, with mask): fp16_conv_dgrad_wf_ex
# with the addend on every s-th row and column
STRIDED = [
    (2, 256, 14, 14, 128, 1, 1, 0, 2, False),   # pointwise kernel (the conv3_x block input)
    (2, 256, 15, 13, 64, 1, 1, 0, 2, False),    # pointwise, odd sides (ceil grid)
    (2, 512, 14, 14, 256, 1, 1, 0, 2, False),   # register-direct kernel (the conv4_x block input)
    (2, 1024, 7, 7, 512, 1, 1, 0, 2, False),    # DMA-staged kernel (the conv5_x block input)
    (2, 16, 9, 9, 24, 3, 1, 1, 3, False),       # LDS-staged kernel, stride 3
    (2, 64, 14, 14, 64, 3, 2, 1, 2, False),     # stride phases of the data gradient itself
    (2, 256, 14, 14, 128, 1, 1, 0, 2, True),    # with a mask over the strided addend
    (2, 512, 10, 10, 256, 1, 1, 0, 2, True),
    (3, 1024, 40, 40, 256, 1, 1, 0, 2, False),  # register-direct kernel over many tiles
    (32, 256, 56, 56, 128, 1, 1, 0, 2, False),  # the conv3_x block input gradient at batch 32
]


@pytest.mark.parametrize("case", STRIDED, ids=[str(c) for c in STRIDED])
def test_strided_addend(case):
    require_gpu()
    n, c, h, w, k, r, st, pad, s, with_mask = case
    d = F.conv_desc(n, c, h, w, k, r, r, st, pad)
    p, q = F.fp16_conv_out_dims(d)
    ah, aw = -(-h // s), -(-w // s)
    seed = 190 + c + k + s
    dy = synth.normal_f16((n, p, q, k), 1e-2, seed, 1)
    wt = synth.normal_f16((k, r, r, c), synth.he_std(c * r * r), seed, 2)
    ad = synth.normal_f16((n, ah, aw, c), 1e-2, seed, 3)
    mask = np.random.default_rng(seed).integers(0, 256, size=ad.size // 8, dtype=np.uint8)
    adm = np.where(_bits(mask, ad.size).reshape(ad.shape), ad, np.float16(0.0)) if with_mask else ad
    full = np.zeros((n, h, w, c), np.float16)
    full[:, ::s, ::s, :] = adm
    DY, W, AD, FULL = dev(dy), dev(wt), dev(ad), dev(full)
    M = torch.from_numpy(mask).to("cuda") if with_mask else None
    WF = torch.empty(F.fp16_conv_dgrad_filter_bytes(d) // 2, dtype=torch.float16, device="cuda")
    ws = F.workspace(F.fp16_conv_workspace_bytes(d, F.PASS_DGRAD))
    note(f"[gpu] dgrad_wf_ex {case}")
    F.fp16_conv_dgrad_filter(d, W, WF)
    ref = torch.empty_like(FULL)
    F.fp16_conv_dgrad_wf(d, DY, WF, FULL, ref, ws)
    DX = torch.full_like(FULL, float("nan"))
    F.fp16_conv_dgrad_wf_ex(d, DY, WF, AD, M, s, DX, ws)
    torch.cuda.synchronize()
    got = host(DX)
    assert np.array_equal(got.view(np.uint16), host(ref).view(np.uint16))
    if n * h * w * c <= 1 << 20:
        shp = oracle.conv_shape(n, c, h, w, k, r, r, st, pad)
        want64, _ = oracle.conv_dgrad_add(shp, dy, wt, full)
        check_close(got, want64, what=f"dgrad_wf_ex {case}")
