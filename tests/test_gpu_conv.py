"""GPU parity of fp16_conv_fwd / fp16_conv_dgrad / fp16_conv_wgrad against the
oracle's float64 convolutions (ResNet-50's convolutions, Section 5.1; FP16
storage with one rounding per output, Section 5.2).

Bar: max |gpu - oracle| <= 1e-2 * RMS(oracle) on every output element, at
sizes the oracle evaluates whole; on sampled outputs for full-size layers;
bit-exact where the sums are exact (delta filters, one-hot gradients)."""

import itertools

import numpy as np
import pytest
import torch

import paper_1911_07384_amd as F
from gpu_util import ConvCase, check_close, dev, host, note, require_gpu, ulp_dist

pytestmark = pytest.mark.gpu

PASSES = ("fwd", "dgrad", "wgrad")

# (n, c, h, w, k, r, s, stride, pad, layout)
SHAPES = [
    (2, 64, 56, 56, 64, 3, 3, 1, 1, "NHWC"),    # the single 3x3 layer, N = 2 (full size)
    (2, 64, 28, 28, 64, 3, 3, 1, 1, "NHWC"),    # several M tiles and a ragged last tile
    (2, 256, 14, 14, 64, 1, 1, 1, 0, "NHWC"),   # bottleneck-entry 1x1
    (2, 64, 14, 14, 256, 1, 1, 1, 0, "NHWC"),   # bottleneck-exit 1x1
    (2, 64, 15, 15, 128, 1, 1, 2, 0, "NHWC"),   # strided 1x1 shortcut, odd size
    (2, 32, 17, 17, 48, 3, 3, 2, 1, "NHWC"),    # strided 3x3, odd size
    (2, 3, 32, 32, 64, 7, 7, 2, 3, "NHWC"),     # the stem (3 input channels): stem kernel, one wave
    (1, 3, 224, 224, 64, 7, 7, 2, 3, "NHWC"),   # the ResNet-50 stem at full size: 7 waves per tile
    (2, 3, 40, 32, 64, 7, 7, 2, 3, "NHWC"),     # stem kernel, 20 output rows: a partial last tile
    (2, 24, 9, 11, 40, 3, 3, 1, 1, "NHWC"),     # channels not a tile multiple
    (3, 16, 6, 5, 3, 3, 3, 1, 2, "NHWC"),       # 3 output channels, pad > R/2
    (4, 512, 1, 1, 200, 1, 1, 1, 0, "NHWC"),    # fully connected as a 1x1 on 1x1 images
                                                # (forward: the reduction in two splits)
    (128, 2048, 1, 1, 1000, 1, 1, 1, 0, "NHWC"),  # the ResNet-50 classifier: 8 splits forward,
                                                  # 4 in the data gradient
    (3, 1000, 1, 1, 600, 1, 1, 1, 0, "NHWC"),   # split reductions with a ragged last split,
                                                # ragged row and channel tiles
    (1, 8, 1, 1, 8, 1, 1, 1, 0, "NHWC"),        # smallest case
    (2, 128, 7, 7, 128, 3, 3, 1, 1, "NHWC"),    # wide channels, tiny image
    (1, 16, 9, 9, 16, 3, 3, 3, 0, "NHWC"),      # stride 3 (9 dgrad phases)
    (2, 64, 12, 12, 64, 3, 3, 1, 1, "NCHW"),
    (2, 3, 20, 20, 16, 7, 7, 2, 3, "NCHW"),
    (2, 64, 15, 15, 128, 1, 1, 2, 0, "NCHW"),
    (2, 64, 15, 15, 64, 3, 3, 2, 1, "NHWC"),    # strided 3x3 on the DMA-staged kernel (fwd)
    (2, 256, 9, 9, 192, 3, 3, 2, 1, "NHWC"),    # dgrad phases of up to 4 taps x 192: DMA-staged; ragged N
    (2, 1024, 5, 5, 96, 1, 1, 1, 0, "NHWC"),    # 1x1 with a 1024-long reduction: DMA-staged
    (2, 512, 7, 7, 128, 1, 1, 1, 0, "NHWC"),    # 1x1 with a 512-long reduction: DMA-staged fwd
    (2, 128, 7, 9, 512, 1, 1, 1, 0, "NHWC"),    # ... and DMA-staged data gradient
    (2, 24, 9, 9, 64, 3, 3, 1, 1, "NHWC"),      # wgrad: 8-channel chunks of one 64-column block span taps
    (2, 8, 12, 12, 128, 1, 1, 2, 0, "NHWC"),    # wgrad: 8 channels, K = 128
    (2, 64, 20, 20, 192, 1, 1, 1, 0, "NHWC"),   # pointwise fwd: 64 -> 192, second channel tile partial
    (3, 128, 9, 9, 384, 1, 1, 1, 0, "NHWC"),    # pointwise fwd over 128 channels, M = 243 (ragged)
    (3, 136, 9, 9, 64, 1, 1, 1, 0, "NHWC"),     # pointwise dgrad: 64 -> 136 channels (one 8-wide chunk
                                                # in the second channel tile)
    (5, 64, 56, 56, 256, 1, 1, 1, 0, "NHWC"),   # pointwise fwd / dgrad over many tiles per workgroup
    (2, 256, 14, 14, 384, 1, 1, 1, 0, "NHWC"),  # pointwise fwd over 256 channels, 3 channel tiles
    (2, 136, 9, 9, 256, 1, 1, 1, 0, "NHWC"),    # pointwise dgrad over 256: 136 outputs (ragged tile)
    (3, 256, 40, 40, 1024, 1, 1, 1, 0, "NHWC"), # pointwise over 256, 38 tiles on 32 row groups
    (5, 256, 28, 28, 200, 1, 1, 2, 0, "NHWC"),  # strided pointwise fwd over 256, ragged channels
    # 3x3 stride 1 on the DMA-staged kernel at its edges:
    (2, 64, 31, 31, 128, 3, 3, 1, 1, "NHWC"),   # odd row width, one 64-channel k-block per tap
    (3, 192, 5, 9, 136, 3, 3, 1, 1, "NHWC"),    # three k-blocks per tap, ragged second N tile
    (2, 128, 1, 13, 128, 3, 3, 1, 1, "NHWC"),   # one-row images: the outer tap rows all padding
    (1, 256, 14, 14, 256, 3, 3, 1, 1, "NHWC"),  # the conv4_x 3x3 layer at N = 1
    (2, 64, 8, 32, 128, 3, 3, 1, 1, "NHWC"),    # 32-pixel rows
]


def _id(s):
    return "n{}c{}h{}w{}k{}r{}s{}st{}p{}{}".format(*s)


@pytest.mark.parametrize("shape", SHAPES, ids=[_id(s) for s in SHAPES])
@pytest.mark.parametrize("which", PASSES)
def test_parity_full(shape, which):
    require_gpu()
    n, c, h, w, k, r, s, st, pad, lay = shape
    case = ConvCase(n, c, h, w, k, r, s, st, pad, lay, seed=1)
    got = case.run(which)
    ref64, ref16 = case.oracle(which)
    check_close(got, ref64, what=f"{which} {case.label}")
    # nearly every element is the oracle's rounding or its neighbour
    assert np.mean(ulp_dist(got, ref16) <= 1) > 0.99


@pytest.mark.parametrize("which", PASSES)
def test_deterministic(which):
    require_gpu()
    case = ConvCase(2, 64, 28, 28, 64, 3, 3, 1, 1, seed=2)
    a = case.run(which)
    b = case.run(which)
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))


# weight gradients split for fewer workgroups (fp16_conv_wgrad_ex): the 3x3
# 64-channel layer, a 1x1 with many filter tiles, the stem (space-to-depth
# path) and a strided 3x3
WG_SHAPES = [(2, 64, 28, 28, 64, 3, 3, 1, 1, "NHWC"), (2, 512, 7, 7, 256, 1, 1, 1, 0, "NHWC"),
             (2, 3, 32, 32, 64, 7, 7, 2, 3, "NHWC"), (2, 64, 15, 15, 128, 3, 3, 2, 1, "NHWC")]


@pytest.mark.parametrize("shape", WG_SHAPES, ids=[_id(s) for s in WG_SHAPES])
def test_wgrad_workgroup_targets(shape):
    require_gpu()
    case = ConvCase(*shape, seed=3)
    ref64, ref16 = case.oracle("wgrad")
    default = case.run("wgrad")
    assert np.array_equal(case.run("wgrad", workgroups=0).view(np.uint16), default.view(np.uint16))
    for wg in (1, 7, 64, 256, 512):
        got = case.run("wgrad", workgroups=wg)
        check_close(got, ref64, what=f"wgrad workgroups={wg} {case.label}")
        assert np.mean(ulp_dist(got, ref16) <= 1) > 0.99
        # deterministic for a given count
        assert np.array_equal(case.run("wgrad", workgroups=wg).view(np.uint16), got.view(np.uint16))
    # the default is 512
    assert np.array_equal(case.run("wgrad", workgroups=512).view(np.uint16),
                          default.view(np.uint16))


@pytest.mark.parametrize("layout", ["NHWC", "NCHW"])
@pytest.mark.parametrize("r,shift", [(3, (0, 0)), (3, (1, -1)), (1, (0, 0)), (7, (-2, 3))])
def test_delta_filter_forward_is_exact(layout, r, shift):
    require_gpu()
    n, c, h, w = 2, 16, 10, 9
    pad = r // 2
    Wk = np.zeros((c, c, r, r), np.float16)
    for ci in range(c):
        Wk[ci, ci, pad + shift[0], pad + shift[1]] = 1.0
    wt = Wk if layout == "NCHW" else np.ascontiguousarray(np.transpose(Wk, (0, 2, 3, 1)))
    case = ConvCase(n, c, h, w, c, r, r, 1, pad, layout, seed=3, wt=wt)
    got = case.run("fwd")
    _, ref16 = case.oracle("fwd")
    assert np.array_equal(got.view(np.uint16), ref16.view(np.uint16))


@pytest.mark.parametrize("r,st,pad", [(3, 1, 1), (3, 2, 1), (1, 2, 0), (7, 2, 3)])
def test_one_hot_gradient_is_exact(r, st, pad):
    require_gpu()
    n, c, h, w, k = 2, 8, 11, 10, 16
    case = ConvCase(n, c, h, w, k, r, r, st, pad, "NHWC", seed=4)
    dy = np.zeros(case.ys, np.float16)
    for (n0, p0, q0, k0) in [(1, case.P - 1, 0, 3), (0, case.P // 2, case.Q - 1, 15)]:
        dy[n0, p0, q0, k0] = 1.0
    case.dy = dy
    for which in ("dgrad", "wgrad"):
        got = case.run(which)
        _, ref16 = case.oracle(which)
        assert np.array_equal(got.astype(np.float64), ref16.astype(np.float64)), which


# The bottleneck block of ResNet-50 stage conv2_x at the paper's per-GPU
# batch of 32 (Section 5.2), layer by layer at full size: sampled outputs.
BLOCK = [
    (32, 256, 56, 56, 64, 1, 1, 1, 0),
    (32, 64, 56, 56, 64, 3, 3, 1, 1),
    (32, 64, 56, 56, 256, 1, 1, 1, 0),
]


@pytest.mark.parametrize("shape", BLOCK, ids=[_id(s + ("NHWC",)) for s in BLOCK])
@pytest.mark.parametrize("which", PASSES)
def test_parity_full_size_sampled(shape, which):
    require_gpu()
    case = ConvCase(*shape, "NHWC", seed=0, dy_std=1e-3)
    got = case.run(which).reshape(-1)
    rng = np.random.default_rng(7)
    idx = np.unique(np.concatenate([rng.integers(0, got.size, 2000), [0, got.size - 1]]))
    ref = case.oracle_at(which, idx)
    rms = np.sqrt(np.mean(ref ** 2))
    err = np.max(np.abs(got[idx].astype(np.float64) - ref))
    assert err <= 1e-2 * rms, (err, rms)
    assert np.all(np.isfinite(got.astype(np.float32)))


# (n, c, h, k): 1x1 stride-1 data gradients plus an addend (the bottleneck's
# first convolution, whose input gradient joins the shortcut's)
ADD_SHAPES = [(2, 256, 14, 64), (3, 136, 9, 64), (2, 64, 28, 64), (4, 256, 56, 64),
              (2, 512, 14, 256), (3, 200, 20, 256), (3, 1024, 40, 256),  # (256-long reductions)
              (128, 2048, 1, 1000)]  # the classifier's data gradient, split reduction + addend


@pytest.mark.parametrize("shape", ADD_SHAPES, ids=["n{}c{}h{}k{}".format(*s) for s in ADD_SHAPES])
def test_dgrad_add_parity(shape):
    require_gpu()
    import oracle
    from paper_1911_07384_amd import synth
    n, c, h, k = shape
    case = ConvCase(n, c, h, h, k, 1, 1, 1, 0, seed=4)
    addend = synth.normal_f16(case.xs, 1e-2, 4, 9)
    ws = F.workspace(F.fp16_conv_workspace_bytes(case.desc, F.PASS_DGRAD))
    out = torch.empty(case.xs, dtype=torch.float16, device="cuda")
    note(f"[gpu] dgrad_add {case.label}")
    F.fp16_conv_dgrad_add(case.desc, dev(case.dy), dev(case.w), dev(addend), out, ws)
    torch.cuda.synchronize()
    got = host(out)
    ref64, ref16 = oracle.conv_dgrad_add(case.shp, case.dy, case.w, addend)
    check_close(got, ref64, what=f"dgrad_add {case.label}")
    assert np.mean(ulp_dist(got, ref16) <= 1) > 0.99


# the data gradient from a filter rearranged ahead of time equals the one-call
# data gradient bit for bit (with and without the addend)
WF_SHAPES = [  # (n, c, h, w, k, r, stride, pad)
    (2, 64, 28, 28, 64, 3, 1, 1),     # the 64-channel 3x3 kernel
    (2, 128, 14, 14, 128, 3, 1, 1),   # DMA-staged kernel
    (2, 64, 15, 15, 128, 1, 2, 0),    # strided 1x1: four phases, three of them empty
    (2, 32, 17, 17, 48, 3, 2, 1),     # strided 3x3: four phases of 1-4 taps
    (3, 16, 6, 5, 3, 3, 1, 2),        # 3 output channels, padded to 8 in the filter
    (2, 64, 14, 14, 256, 1, 1, 0),    # pointwise kernel (64 -> 256 data gradient)
]


@pytest.mark.parametrize("shape", WF_SHAPES, ids=[str(s) for s in WF_SHAPES])
@pytest.mark.parametrize("with_addend", [False, True])
def test_dgrad_from_rearranged_filter_is_identical(shape, with_addend):
    require_gpu()
    from paper_1911_07384_amd import synth
    n, c, h, w, k, r, st, pad = shape
    case = ConvCase(n, c, h, w, k, r, r, st, pad, seed=5)
    ws = F.workspace(F.fp16_conv_workspace_bytes(case.desc, F.PASS_DGRAD))
    wf = F.workspace(F.fp16_conv_dgrad_filter_bytes(case.desc))
    addend = dev(synth.normal_f16(case.xs, 1e-2, 5, 9)) if with_addend else None
    a = torch.empty(case.xs, dtype=torch.float16, device="cuda")
    b = torch.empty_like(a)
    note(f"[gpu] dgrad_wf {case.label} addend={with_addend}")
    if with_addend:
        F.fp16_conv_dgrad_add(case.desc, dev(case.dy), dev(case.w), addend, a, ws)
    else:
        F.fp16_conv_dgrad(case.desc, dev(case.dy), dev(case.w), a, ws)
    F.fp16_conv_dgrad_filter(case.desc, dev(case.w), wf)
    F.fp16_conv_dgrad_wf(case.desc, dev(case.dy), wf, addend, b, ws)
    torch.cuda.synchronize()
    assert np.array_equal(host(a).view(np.uint16), host(b).view(np.uint16))


def test_batched_filter_rearrangement_is_identical():
    # every ResNet-50 filter shape (and the classifier as a 1x1 convolution,
    # K = 1000) plus ragged and strided ones: 70 filters, so the batch spans
    # three launches; each wf must equal the one-filter call's bit for bit
    require_gpu()
    from paper_1911_07384_amd import resnet50, synth
    shapes = [(L.c, L.k, L.r, L.stride) for L in resnet50.LAYERS]
    shapes += [(2048, 1000, 1, 1), (24, 40, 3, 1), (8, 8, 5, 2), (136, 72, 3, 2), (3, 64, 7, 2)]
    shapes = (shapes * 3)[:70]
    descs, ws, wb, wa = [], [], [], []
    for i, (c, k, r, st) in enumerate(shapes):
        d = F.conv_desc(2, c, 16, 16, k, r, r, st, r // 2)
        descs.append(d)
        ws.append(dev(synth.normal_f16((k, r, r, c), 0.1, 11, i)))
        nb = F.fp16_conv_dgrad_filter_bytes(d) // 2
        wa.append(torch.full((nb,), float("nan"), dtype=torch.float16, device="cuda"))
        wb.append(torch.full((nb,), float("nan"), dtype=torch.float16, device="cuda"))
    note(f"[gpu] dgrad_filters x{len(descs)}")
    F.fp16_conv_dgrad_filters(descs, ws, wb)
    for d, w, a in zip(descs, ws, wa):
        F.fp16_conv_dgrad_filter(d, w, a)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(wa, wb)):
        assert np.array_equal(host(a).view(np.uint16), host(b).view(np.uint16)), shapes[i]
