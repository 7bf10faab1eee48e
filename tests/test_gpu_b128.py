"""Parity at the full batch of the measured workloads (ResNet-50, Section 5.1,
batch 128; all-FP16 storage, Section 5.2).

1. Every distinct ResNet-50 convolution shape (23 shapes, the 53 layers) at
   batch 128, forward, data gradient and weight gradient through the C ABI
   -- the very calls, and so the very kernel variants (staging depth, tile
   widths, split counts), that the per-layer sweep times -- against the
   oracle on 2,000 sampled outputs per pass plus the first and the last:
   max|err| <= 1e-2 * RMS of the sampled reference values.
2. One training step of the whole network at batch 128 on 224x224 images,
   teacher-forced: a set of its calls covering every kind of call, every
   stage, both strides, the downsampling shortcuts, the stem, the pools, the
   classifier and the loss, each replayed through the oracle on the inputs
   the GPU call saw.  Convolutions on sampled outputs at the bar above; the
   fused BN apply bit-exact against the declared float32 apply with the
   statistics the call wrote, and at the own-statistics bar of test_gpu_bn
   (1 ulp, or 2^-22 (1 + |s beta| + |r|) absolute) against the oracle's BN; BN
   backward, pools and loss on every element at the single-operation bars of
   test_gpu_network.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import dev, host, note, require_gpu, ulp_dist
from test_gpu_network import masked_addend
from paper_1911_07384_amd import resnet50, synth
import paper_1911_07384_amd as F

pytestmark = pytest.mark.gpu

N = 128
NSAMP = 2000


def _sample_idx(size, nsamp, seed):
    rng = np.random.default_rng(seed)
    idx = rng.choice(size, min(nsamp, size), replace=False)
    return np.unique(np.concatenate([idx, [0, size - 1]])).astype(np.int64)


def _close_sampled(got, ref, what):
    g = got.astype(np.float64)
    assert np.all(np.isfinite(g)), what
    rms = float(np.sqrt(np.mean(ref ** 2)))
    err = float(np.max(np.abs(g - ref)))
    assert err <= 1e-2 * rms, f"{what}: max err {err:.3e} > 1e-2 * RMS {rms:.3e}"


@pytest.mark.parametrize("li", range(len(resnet50.LAYERS)),
                         ids=[l.name.replace(" ", "") for l in resnet50.LAYERS])
def test_resnet50_layer_b128_sampled(li):
    require_gpu()
    L = resnet50.LAYERS[li]
    p = L.out_hw
    seed = 60 + li
    x = synth.normal_f16((N, L.hw, L.hw, L.c), 1.0, seed, 1)
    w = synth.normal_f16((L.k, L.r, L.r, L.c), synth.he_std(L.c * L.r * L.r), seed, 2)
    dy = synth.normal_f16((N, p, p, L.k), 1e-3, seed, 3)
    d = F.conv_desc(N, L.c, L.hw, L.hw, L.k, L.r, L.r, L.stride, L.pad)
    assert F.fp16_conv_out_dims(d) == (p, p)
    shp = oracle.conv_shape(N, L.c, L.hw, L.hw, L.k, L.r, L.r, L.stride, L.pad)
    X, W, DY = dev(x), dev(w), dev(dy)
    ws = F.workspace(max(F.fp16_conv_workspace_bytes(d, q) for q in (0, 1, 2)))
    y = torch.empty((N, p, p, L.k), dtype=torch.float16, device="cuda")
    dx = torch.empty_like(X)
    dw = torch.empty_like(W)
    note(f"[gpu] b128 {L.name} fwd/dgrad/wgrad")
    F.fp16_conv_fwd(d, X, W, y, ws)
    F.fp16_conv_dgrad(d, DY, W, dx, ws)
    F.fp16_conv_wgrad(d, X, DY, dw, ws)
    torch.cuda.synchronize()
    for which, out, fn, a, b in (("fwd", y, oracle.conv_fwd_at, x, w),
                                 ("dgrad", dx, oracle.conv_dgrad_at, dy, w),
                                 ("wgrad", dw, oracle.conv_wgrad_at, x, dy)):
        got = host(out).reshape(-1)
        idx = _sample_idx(got.size, NSAMP, seed * 7 + len(which))
        _close_sampled(got[idx], fn(shp, a, b, idx), f"{L.name} {which} N=128")


# ---- the whole step at batch 128 ----------------------------------------------

# the blocks checked: the first of each stage (stride 2 from stage 2 on, with
# the downsampling shortcut), a stride-1 block of stages 2 and 3, the last block
BLOCKS = ("l1.0", "l2.0", "l2.1", "l3.0", "l3.1", "l4.0", "l4.2")
OTHER = ("stem", "stem.bn", "pool", "gap", "fc", "loss")


def _group(op):
    """The checked group of a call of the step, or None."""
    base = op.a.get("conv", op.name)
    for b in BLOCKS:
        if op.name.startswith(b + ".") or base.startswith(b + "."):
            return b
    if op.name in OTHER or base in OTHER:
        return "stem+pool+head"
    return None


@pytest.fixture(scope="module")
def net_b128():
    require_gpu()
    from paper_1911_07384_amd.network import ResNet50
    net = ResNet50(n=N, image=224, seed=7)
    net.load_batch(7)
    note("[gpu] resnet50 n=128 224x224 forward+backward")
    # the data-gradient filters are rearranged during the forward, as in the step
    net.forward()
    net.backward()
    torch.cuda.synchronize()
    yield net
    del net
    torch.cuda.empty_cache()


class _Host(dict):
    """Host copies of the network's buffers, fetched on first use."""

    def __init__(self, net):
        super().__init__()
        self.net = net

    def __missing__(self, key):
        v = host(self.net.buffers[key]).copy()
        self[key] = v
        return v


def _conv_sampled(op, H, seed):
    a = op.a
    d = a["desc"]
    shp = oracle.conv_shape(d.n, d.c, d.h, d.w, d.k, d.r, d.s, (d.stride_h, d.stride_w),
                            (d.pad_h, d.pad_w), "NHWC")
    k = op.kind
    if k in ("conv_fwd", "conv_bn_fwd"):
        got = H[a["y"]].reshape(-1)
        idx = _sample_idx(got.size, 500, seed)
        ref = oracle.conv_fwd_at(shp, H[a["x"]], H[a["w"]], idx)
    elif k == "conv_dgrad":
        got = H[a["dx"]].reshape(-1)
        idx = _sample_idx(got.size, 500, seed)
        ref = oracle.conv_dgrad_at(shp, H[a["dy"]], H[a["w"]], idx)
    elif k == "conv_dgrad_add":
        got = H[a["dx"]].reshape(-1)
        idx = _sample_idx(got.size, 500, seed)
        ref = oracle.conv_dgrad_at(shp, H[a["dy"]], H[a["w"]], idx) + \
            masked_addend(a, H).reshape(-1)[idx].astype(np.float64)
    else:
        got = H[a["dw"]].reshape(-1)
        idx = _sample_idx(got.size, 500, seed)
        ref = oracle.conv_wgrad_at(shp, H[a["x"]], H[a["dy"]], idx)
    _close_sampled(got[idx], ref, f"{op.name}:{k} N=128")


def _bn_apply_checks(op, H):
    a = op.a
    d = a["bn"]
    shp = oracle.bn_shape(d.n, d.c, d.h, d.w)
    res = None if a["res"] is None else H[a["res"]]
    g, b = H[op.name + ".gamma"], H[op.name + ".beta"]
    st = H[a["stats"]]
    want = oracle.bn_apply_f32(shp, H[a["y"]], g, b, st[:d.c], st[d.c:], res, d.post_scale,
                               bool(d.relu), swap=bool(d.swap))
    assert np.array_equal(H[a["z"]].view(np.uint16), want.view(np.uint16)), op.name
    ref = oracle.bn_fwd(shp, H[a["y"]], g, b, res, d.eps, d.post_scale, bool(d.relu),
                        swap=bool(d.swap))
    # own statistics: 1 ulp, or (where the shortcut nearly cancels the BN term
    # and the result's ulp is small) the float32 statistics' absolute error
    z = H[a["z"]]
    absd = np.abs(z.astype(np.float64) - ref["y"].astype(np.float64))
    bound = 2.0 ** -22 * (1 + np.abs(d.post_scale * b.astype(np.float64)).max()
                          + (np.abs(res.astype(np.float64)) if res is not None else 0))
    assert np.all((ulp_dist(z, ref["y"]) <= 1) | (absd <= bound)), op.name


@pytest.mark.parametrize("group", ("stem+pool+head",) + BLOCKS)
def test_resnet50_step_b128_teacher_forced(net_b128, group):
    from test_gpu_network import _check_op
    net = net_b128
    kinds = set()
    for i, op in enumerate(net.fwd + net.bwd):
        if _group(op) != group:
            continue
        H = _Host(net)
        note(f"[check] {op.name}:{op.kind}")
        if op.kind.startswith("conv"):
            _conv_sampled(op, H, 1000 + i)
            if op.kind == "conv_bn_fwd":
                _bn_apply_checks(op, H)
        else:
            _check_op(net, op, H)
        kinds.add(op.kind)
        del H
    if group == "stem+pool+head":
        assert {"bn_maxpool_fwd", "maxpool_bwd", "avgpool_fwd", "avgpool_bwd",
                "softmax_ce", "bn_bwd", "conv_wgrad", "conv_fwd", "conv_dgrad"} <= kinds, kinds
    else:
        assert {"conv_bn_fwd", "bn_bwd", "conv_wgrad", "conv_dgrad_add"} <= kinds, kinds
