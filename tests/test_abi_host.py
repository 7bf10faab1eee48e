"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/fp16train.h declares, and rejects invalid arguments
with the documented status before anything is launched.  Pointers here are
fake addresses that validation must reject without dereferencing: every call
here carries at least one invalid argument, so nothing is ever launched."""

import ctypes
import os
import re

import pytest

import paper_1911_07384_amd as F

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "fp16train.h")

OK, NULL, SHAPE, LAYOUT, MISALIGNED, ALIASING, WORKSPACE = 0, 1, 2, 3, 4, 5, 6


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fp16_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_function():
    names = _declared()
    assert "fp16_conv_fwd" in names and "fp16_sgd_step" in names and len(names) >= 11
    lib = ctypes.CDLL(F.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(F.EXPORTS) == set(names)


def test_version_and_status_strings():
    assert F.fp16_version().startswith("fp16train")
    for s in range(9):
        assert F.fp16_status_string(s)
    assert F.fp16_status_string(99) == "unknown status"


def _conv(**kw):
    base = dict(n=2, c=64, h=56, w=56, k=64, r=3, s=3, stride=1, pad=1, layout="NHWC")
    base.update(kw)
    return F.conv_desc(base["n"], base["c"], base["h"], base["w"], base["k"], base["r"], base["s"],
                       base["stride"], base["pad"], base["layout"])


def _call(fn, desc, a, b, c, ws=0, wsb=0):
    return getattr(F.lib(), fn)(ctypes.byref(desc) if desc is not None else None, a, b, c, ws, wsb,
                                None)


A = 0x10000000  # fake, 16-byte aligned, far apart
B = 0x20000000
Cc = 0x30000000
WS = 0x40000000


@pytest.mark.parametrize("fn", ["fp16_conv_fwd", "fp16_conv_dgrad", "fp16_conv_wgrad"])
def test_conv_validation(fn):
    d = _conv()
    assert _call(fn, None, A, B, Cc) == NULL
    assert _call(fn, d, None, B, Cc) == NULL
    assert _call(fn, d, A, B, None) == NULL
    # NCHW is accepted; it needs staging workspace, whose absence is the error
    assert _call(fn, _conv(layout=1), A, B, Cc) == WORKSPACE
    bad = _conv()
    bad.layout = 7
    assert _call(fn, bad, A, B, Cc) == LAYOUT
    for field, val in [("n", 0), ("c", 0), ("h", -1), ("k", 0), ("stride_h", 0), ("pad_w", -1),
                       ("r", 100)]:
        d2 = _conv()
        setattr(d2, field, val)
        assert _call(fn, d2, A, B, Cc) == SHAPE, field
    # kernel larger than the padded image
    assert _call(fn, _conv(h=1, w=1, pad=0), A, B, Cc) == SHAPE
    assert _call(fn, d, A + 2, B, Cc) == MISALIGNED
    assert _call(fn, d, A, B, Cc + 8) == MISALIGNED


def test_wgrad_workgroup_target_validation():
    lib = F.lib()
    d = _conv()
    need = F.fp16_conv_workspace_bytes(d, F.PASS_WGRAD)
    f = lambda wg, x=A: lib.fp16_conv_wgrad_ex(ctypes.byref(d), x, B, Cc, WS, need, wg, None)
    assert f(-1) == SHAPE and f(513) == SHAPE
    assert f(0, None) == NULL and f(256, None) == NULL
    # dw over the workspace, at any target
    for wg in (0, 1, 512):
        assert lib.fp16_conv_wgrad_ex(ctypes.byref(d), A, B, WS + 64, WS, need, wg, None) == ALIASING


def test_conv_workspace_and_aliasing():
    d = _conv()
    # native NHWC forward with C % 8 == 0 needs no workspace ...
    assert F.fp16_conv_workspace_bytes(d, F.PASS_FWD) == 0
    # ... so overlapping output/input is the next check
    assert _call("fp16_conv_fwd", d, A, B, A + 64) == ALIASING
    # the data gradient needs its phase filters and the weight gradient its partials
    for p in (F.PASS_DGRAD, F.PASS_WGRAD):
        need = F.fp16_conv_workspace_bytes(d, p)
        assert need > 0
    need = F.fp16_conv_workspace_bytes(d, F.PASS_WGRAD)
    assert _call("fp16_conv_wgrad", d, A, B, Cc, 0, 0) == WORKSPACE
    assert _call("fp16_conv_wgrad", d, A, B, Cc, WS, need - 1) == WORKSPACE
    assert _call("fp16_conv_wgrad", d, A, B, Cc, WS + 4, need) == MISALIGNED
    assert _call("fp16_conv_wgrad", d, A, B, WS + 16, WS, need) == ALIASING
    # channel padding and NCHW need staging space in the forward pass too
    assert F.fp16_conv_workspace_bytes(_conv(c=3), F.PASS_FWD) > 0
    assert F.fp16_conv_workspace_bytes(_conv(layout="NCHW"), F.PASS_FWD) > 0
    assert F.fp16_conv_workspace_bytes(_conv(), 5) == 0


def test_dgrad_filter_validation():
    d = _conv()
    lib = F.lib()
    # bytes: C x R x S x K (K padded to 8); NCHW is not offered
    assert F.fp16_conv_dgrad_filter_bytes(d) == 64 * 3 * 3 * 64 * 2
    assert F.fp16_conv_dgrad_filter_bytes(_conv(k=3)) == 64 * 3 * 3 * 8 * 2
    assert F.fp16_conv_dgrad_filter_bytes(_conv(layout="NCHW")) == 0
    f = lib.fp16_conv_dgrad_filter
    assert f(None, A, B, None) == NULL
    assert f(ctypes.byref(d), None, B, None) == NULL
    assert f(ctypes.byref(d), A, None, None) == NULL
    assert f(ctypes.byref(_conv(layout="NCHW")), A, B, None) == UNSUPPORTED
    assert f(ctypes.byref(d), A + 2, B, None) == MISALIGNED
    assert f(ctypes.byref(d), A, A + 64, None) == ALIASING
    g = lib.fp16_conv_dgrad_wf
    need = F.fp16_conv_workspace_bytes(d, F.PASS_DGRAD)
    assert g(ctypes.byref(d), None, B, None, Cc, WS, need, None) == NULL
    assert g(ctypes.byref(d), A, None, None, Cc, WS, need, None) == NULL
    assert g(ctypes.byref(_conv(layout="NCHW")), A, B, None, Cc, WS, 1 << 30, None) == UNSUPPORTED
    assert g(ctypes.byref(d), A, B, None, Cc, WS + 4, need, None) == MISALIGNED
    assert g(ctypes.byref(d), A, B, None, Cc, 0, 0, None) == WORKSPACE
    # dx over the rearranged filter
    assert g(ctypes.byref(d), A, B, None, B + 64, WS, need, None) == ALIASING
    # the addend under a ReLU mask: dy, wf, addend, mask, dx, ws
    gm = lib.fp16_conv_dgrad_wf_m
    M = Cc + (16 << 20)
    ok = [A, B, Cc + (8 << 20), M, Cc, WS, need, None]
    assert gm(ctypes.byref(d), *ok[:2], None, *ok[3:]) == NULL
    assert gm(ctypes.byref(d), *ok[:3], None, *ok[4:]) == NULL
    assert gm(ctypes.byref(_conv(layout="NCHW")), *ok[:6], 1 << 30, None) == UNSUPPORTED
    assert gm(ctypes.byref(_conv(c=20)), *ok) == UNSUPPORTED  # C % 8 != 0
    for at in (Cc, Cc + 2 * 56 * 56 * 64 * 2 - 8, WS):  # the mask under dx or the workspace
        bad = list(ok)
        bad[3] = at
        assert gm(ctypes.byref(d), *bad) == ALIASING, hex(at)
    assert gm(ctypes.byref(d), *ok[:4], B + 64, WS, need, None) == ALIASING  # dx over wf
    # the strided addend: dy, wf, addend, mask, stride, dx, ws
    ge = lib.fp16_conv_dgrad_wf_ex
    ex = [A, B, Cc + (8 << 20), None, 2, Cc, WS, need, None]
    for bad_s in (0, -1, 17):
        assert ge(ctypes.byref(d), *ex[:4], bad_s, *ex[5:]) == SHAPE
    assert ge(ctypes.byref(d), *ex[:2], None, None, 2, *ex[5:]) == NULL
    assert ge(ctypes.byref(_conv(layout="NCHW")), *ex[:7], 1 << 30, None) == UNSUPPORTED
    assert ge(ctypes.byref(d), *ex[:2], Cc, None, 2, Cc, *ex[6:]) == ALIASING  # addend is dx
    # the addend's own extent (a quarter of dx's at stride 2) over dx's tail
    assert ge(ctypes.byref(d), *ex[:2], Cc + 2 * 56 * 56 * 64 * 2 - 64, None, 2, *ex[5:]) == ALIASING


@pytest.mark.parametrize("hw,r,st,pad", [(56, 3, 1, 1), (56, 1, 2, 0), (224, 7, 2, 3), (7, 3, 1, 1),
                                         (14, 3, 2, 1), (1, 1, 1, 0), (5, 3, 2, 0)])
def test_out_dims(hw, r, st, pad):
    d = _conv(h=hw, w=hw, r=r, s=r, stride=st, pad=pad)
    p, q = F.fp16_conv_out_dims(d)
    assert p == q == (hw + 2 * pad - r) // st + 1


def test_bn_validation():
    lib = F.lib()
    d = F.bn_desc(2, 64, 8, 8)
    need = F.fp16_bn_workspace_bytes(d)
    assert need > 0
    args = [A, B, B + 256, None, Cc, WS + (1 << 20), WS, need, None]
    assert lib.fp16_bn_relu(None, *args) == NULL
    assert lib.fp16_bn_relu(ctypes.byref(d), None, *args[1:]) == NULL
    assert lib.fp16_bn_relu(ctypes.byref(d), A, B, B + 256, None, Cc, None, WS, need, None) == NULL
    assert lib.fp16_bn_relu(ctypes.byref(d), A, B, B + 256, None, Cc, WS + (1 << 20), WS, need - 4,
                            None) == WORKSPACE
    assert lib.fp16_bn_relu(ctypes.byref(d), A + 2, B, B + 256, None, Cc, WS + (1 << 20), WS, need,
                            None) == MISALIGNED
    # y overlapping x partially is rejected (exactly equal is allowed: in place)
    assert lib.fp16_bn_relu(ctypes.byref(d), A, B, B + 256, None, A + 16, WS + (1 << 20), WS, need,
                            None) == ALIASING
    bad = F.bn_desc(2, 64, 8, 8)
    bad.layout = 3
    assert lib.fp16_bn_relu(ctypes.byref(bad), *args) == LAYOUT
    bad = F.bn_desc(0, 64, 8, 8)
    assert lib.fp16_bn_relu(ctypes.byref(bad), *args) == SHAPE
    # backward: required pointers and the dx/dy in-place rule
    bw = [A, None, Cc, B, B + 256, None, WS + (1 << 20), Cc + (1 << 20), B + 512, B + 768, None, WS,
          need, None]
    assert lib.fp16_bn_relu_bwd(ctypes.byref(d), None, *bw[1:]) == NULL
    bw_alias = list(bw)
    bw_alias[7] = Cc + 32  # dx partially overlapping dy
    assert lib.fp16_bn_relu_bwd(ctypes.byref(d), *bw_alias) == ALIASING
    bw_alias = list(bw)
    bw_alias[7] = A  # dx == x
    assert lib.fp16_bn_relu_bwd(ctypes.byref(d), *bw_alias) == ALIASING


def test_bn_workspace_must_not_overlap_inputs():
    # the workspace (partial sums, the kept ReLU mask) is written while the
    # inputs are read: any overlap with them is rejected
    lib = F.lib()
    d = F.bn_desc(2, 64, 8, 8)
    need = F.fp16_bn_workspace_bytes(d)
    ok = [A, B, B + 256, Cc + (2 << 20), Cc, WS + (1 << 20), WS, need, None]
    assert lib.fp16_bn_relu(ctypes.byref(d), *ok[:6], A + 4096, need, None) == ALIASING  # x
    bad = list(ok)
    bad[3] = WS + 256  # residual inside the workspace
    assert lib.fp16_bn_relu(ctypes.byref(d), *bad) == ALIASING
    bad = list(ok)
    bad[6] = B  # workspace over gamma and beta
    assert lib.fp16_bn_relu(ctypes.byref(d), *bad) == ALIASING
    # backward: x, y, dy, residual, gamma, beta, stats
    bw = [A, Cc + (2 << 20), Cc, B, B + 256, Cc + (3 << 20), WS + (1 << 20), Cc + (1 << 20),
          B + 512, B + 768, None, WS, need, None]
    for i, at in ((0, A), (1, Cc + (2 << 20)), (2, Cc), (5, Cc + (3 << 20)), (3, B),
                  (6, WS + (1 << 20))):
        bad = list(bw)
        bad[11] = at  # the workspace placed on input i
        if i == 6:
            bad[6] = WS + 64  # stats inside the workspace
            bad[11] = WS
        assert lib.fp16_bn_relu_bwd(ctypes.byref(d), *bad) == ALIASING, i
    # the fused convolution + BN forward: workspace over x or the filter
    cd = _conv()
    bd = F.bn_desc(cd.n, cd.k, cd.h, cd.w)
    need = F.fp16_conv_bn_workspace_bytes(cd, bd)
    assert need > 0
    args = [A, B, B + (1 << 20), B + (1 << 20) + 256, None, Cc, Cc + (4 << 20), WS + (8 << 20)]
    assert lib.fp16_conv_bn_relu_fwd(ctypes.byref(cd), ctypes.byref(bd), *args, A, need,
                                     None) == ALIASING
    assert lib.fp16_conv_bn_relu_fwd(ctypes.byref(cd), ctypes.byref(bd), *args, B, need,
                                     None) == ALIASING


@pytest.mark.parametrize("fn", ["fp16_sgd_step", "fp16_sgd_step_f16"])
def test_sgd_validation(fn):
    f = getattr(F.lib(), fn)
    assert f(None, None, None, 0, 0.1, 0.9, 1e-4, None) == OK  # n = 0: no-op
    assert f(None, B, Cc, 8, 0.1, 0.9, 1e-4, None) == NULL
    assert f(A + 2, B, Cc, 8, 0.1, 0.9, 1e-4, None) == MISALIGNED
    assert f(A, A + 16, Cc, 64, 0.1, 0.9, 1e-4, None) == ALIASING
    assert f(A, B, A + 64, 64, 0.1, 0.9, 1e-4, None) == ALIASING


@pytest.mark.parametrize("fn", ["fp16_conv_fwd", "fp16_conv_dgrad", "fp16_conv_wgrad"])
def test_conv_accum_validation(fn):
    # binary16 accumulation: only 0 / 1, and only NHWC
    d = _conv()
    d.accum = 2
    assert _call(fn, d, A, B, Cc) == 7
    d = _conv(layout="NCHW")
    d.accum = 1
    assert _call(fn, d, A, B, Cc) == 7
    assert F.fp16_conv_workspace_bytes(d, F.PASS_FWD) == 0  # invalid descriptor


def test_conv_accum_needs_no_workspace():
    # the binary16 chains read and write the caller's tensors only
    d = _conv()
    d.accum = 1
    for pass_ in (F.PASS_FWD, F.PASS_DGRAD, F.PASS_WGRAD):
        assert F.fp16_conv_workspace_bytes(d, pass_) == 0
    assert F.fp16_conv_workspace_bytes(_conv(), F.PASS_WGRAD) > 0


def test_conv_accum_rejects_fused_forms():
    # the strict mode is the plain data gradient only: no addend, no
    # rearranged filter, no fused BN (FP16_ERR_UNSUPPORTED, nothing launched)
    d = _conv()
    d.accum = 1
    l = F.lib()
    assert l.fp16_conv_dgrad_add(ctypes.byref(d), A, B, Cc, Cc + (1 << 20), None, 0, None) == 7
    assert l.fp16_conv_dgrad_wf(ctypes.byref(d), A, B, None, Cc, None, 0, None) == 7
    bd = F.bn_desc(d.n, d.k, d.h, d.w)
    assert F.fp16_conv_bn_workspace_bytes(d, bd) == 0


def test_wgrad_noalloc_validates_before_touching_the_device():
    # no GPU here: every refusal happens before any HIP call
    lib = F.lib()
    assert lib.fp16_noalloc_scratch_bytes() == 32 << 20
    big = F.conv_desc(128, 3, 224, 224, 64, 7, 7, 2, 3)  # the stem at batch 128: 81 MiB
    assert F.fp16_conv_workspace_bytes(big, F.PASS_WGRAD) > lib.fp16_noalloc_scratch_bytes()
    assert lib.fp16_conv_wgrad_noalloc(ctypes.byref(big), A, B, Cc, None) == WORKSPACE
    bad = _conv()
    bad.n = 0
    assert lib.fp16_conv_wgrad_noalloc(ctypes.byref(bad), A, B, Cc, None) == SHAPE
    assert lib.fp16_conv_wgrad_noalloc(None, A, B, Cc, None) == NULL
    assert lib.fp16_conv_wgrad_noalloc(ctypes.byref(_conv()), A, None, Cc, None) == NULL


# ---- pooling and loss: every call below is invalid, nothing is launched ---------

UNSUPPORTED = 7


def _pool(**kw):
    base = dict(n=2, c=64, h=112, w=112, r=3, s=3, stride=2, pad=1, layout="NHWC")
    base.update(kw)
    return F.pool_desc(base["n"], base["c"], base["h"], base["w"], base["r"], base["s"],
                       base["stride"], base["pad"], base["layout"])


def test_pool_out_dims():
    assert F.fp16_pool_out_dims(_pool()) == (56, 56)
    assert F.fp16_pool_out_dims(_pool(h=7, w=7, r=7, s=7, stride=1, pad=0)) == (1, 1)
    for kw in [dict(pad=3), dict(r=16), dict(stride=0), dict(n=0), dict(h=1, w=1, pad=0),
               dict(layout=2)]:
        d = _pool(**{k: v for k, v in kw.items() if k != "layout"})
        if "layout" in kw:
            d.layout = kw["layout"]
        with pytest.raises(F.Fp16Error):
            F.fp16_pool_out_dims(d)


def test_maxpool_validation():
    l = F.lib()
    d = _pool()
    assert l.fp16_maxpool_fwd(None, A, B, Cc, None) == NULL
    assert l.fp16_maxpool_fwd(ctypes.byref(d), A, B, None, None) == NULL
    assert l.fp16_maxpool_fwd(ctypes.byref(d), A, B, Cc + 8, None) == MISALIGNED
    assert l.fp16_maxpool_fwd(ctypes.byref(d), A, A + 16, Cc, None) == ALIASING
    assert l.fp16_maxpool_fwd(ctypes.byref(_pool(pad=3)), A, B, Cc, None) == SHAPE
    assert l.fp16_maxpool_bwd(ctypes.byref(d), None, B, Cc, None) == NULL
    assert l.fp16_maxpool_bwd(ctypes.byref(d), A, B, B + 32, None) == ALIASING
    assert l.fp16_maxpool_bwd(ctypes.byref(d), A + 4, B, Cc, None) == MISALIGNED


def test_avgpool_validation():
    l = F.lib()
    g = _pool(h=7, w=7, r=7, s=7, stride=1, pad=0, c=2048)
    assert l.fp16_avgpool_fwd(ctypes.byref(_pool()), A, B, None) == UNSUPPORTED
    assert l.fp16_avgpool_fwd(ctypes.byref(g), None, B, None) == NULL
    assert l.fp16_avgpool_fwd(ctypes.byref(g), A, A + 64, None) == ALIASING
    assert l.fp16_avgpool_bwd(ctypes.byref(g), A, B + 2, None) == MISALIGNED
    assert l.fp16_avgpool_bwd(ctypes.byref(_pool(h=7, w=7, r=7, s=7, pad=1)), A, B, None) == \
        UNSUPPORTED


def test_softmax_ce_validation():
    l = F.lib()
    D, E, G = 0x50000000, 0x60000000, 0x70000000
    assert l.fp16_softmax_ce(0, 1000, A, B, Cc, D, E, G, None) == SHAPE
    assert l.fp16_softmax_ce(128, 0, A, B, Cc, D, E, G, None) == SHAPE
    assert l.fp16_softmax_ce(128, 70000, A, B, Cc, D, E, G, None) == SHAPE
    assert l.fp16_softmax_ce(128, 1000, A, B, None, D, E, G, None) == NULL
    assert l.fp16_softmax_ce(128, 1000, A, B, Cc, D + 4, E, G, None) == MISALIGNED
    assert l.fp16_softmax_ce(128, 1000, A, B, Cc, D, A + 16, G, None) == ALIASING
    assert l.fp16_softmax_ce(128, 1000, A, B, Cc, D, E, B, None) == ALIASING


def test_bn_swap_needs_residual_and_valid_flag():
    l = F.lib()
    d = F.bn_desc(2, 64, 8, 8, "NHWC", 1e-5, 0.25, True, swap=True)
    WSB = 1 << 20
    # residual NULL with swap: FP16_ERR_NULL before anything else is checked
    assert l.fp16_bn_relu(ctypes.byref(d), A, B, B + 256, None, Cc, WS, WS + 4096, WSB, None) == NULL
    assert l.fp16_bn_relu_bwd(ctypes.byref(d), A, None, B, Cc, Cc + 256, None, WS, A + 4096,
                              Cc + 512, Cc + 768, None, WS + 8192, WSB, None) == NULL
    d.swap = 2
    assert l.fp16_bn_relu(ctypes.byref(d), A, B, B + 256, A + 64, Cc, WS, WS + 4096, WSB,
                          None) == SHAPE


def test_conv_bn_validation():
    l = F.lib()
    cd = F.conv_desc(2, 64, 14, 14, 64, 3, 3, 1, 1)
    bd = F.bn_desc(2, 64, 14, 14, "NHWC", 1e-5, 0.25, True)
    assert F.fp16_conv_bn_workspace_bytes(cd, bd) > 0
    D = 0x50000000
    args = [A, B, Cc, Cc + 256, None, D, D + (1 << 22), WS, WS + (1 << 22), 1 << 20, None]
    # a BN descriptor of another shape
    bad = F.bn_desc(2, 64, 7, 7, "NHWC", 1e-5, 0.25, True)
    assert l.fp16_conv_bn_relu_fwd(ctypes.byref(cd), ctypes.byref(bad), *args) == SHAPE
    # given statistics are not what the fused call computes
    gs = F.bn_desc(2, 64, 14, 14, "NHWC", 1e-5, 0.25, True, use_stats=True)
    assert l.fp16_conv_bn_relu_fwd(ctypes.byref(cd), ctypes.byref(gs), *args) == SHAPE
    # NCHW and channel counts that are not multiples of 8 are not fused
    nchw = F.conv_desc(2, 64, 14, 14, 64, 3, 3, 1, 1, "NCHW")
    assert l.fp16_conv_bn_relu_fwd(ctypes.byref(nchw), ctypes.byref(bd), *args) == UNSUPPORTED
    odd = F.conv_desc(2, 64, 14, 14, 60, 3, 3, 1, 1)
    bodd = F.bn_desc(2, 60, 14, 14, "NHWC", 1e-5, 0.25, True)
    assert l.fp16_conv_bn_relu_fwd(ctypes.byref(odd), ctypes.byref(bodd), *args) == UNSUPPORTED
    # workspace too small, missing pointers, overlapping outputs
    small = list(args)
    small[9] = 16
    assert l.fp16_conv_bn_relu_fwd(ctypes.byref(cd), ctypes.byref(bd), *small) == WORKSPACE
    nul = list(args)
    nul[6] = None
    assert l.fp16_conv_bn_relu_fwd(ctypes.byref(cd), ctypes.byref(bd), *nul) == NULL
    ov = list(args)
    ov[6] = D + 64  # z overlaps y without being y
    assert l.fp16_conv_bn_relu_fwd(ctypes.byref(cd), ctypes.byref(bd), *ov) == ALIASING


def test_kept_mask_validation():
    lib = F.lib()
    d = F.bn_desc(2, 64, 8, 8)
    assert F.fp16_bn_mask_bytes(d) == 2 * 8 * 8 * 64 // 8
    # not offered: NCHW, C/8 not a power of two, no ReLU, the BN swap
    for bad in (F.bn_desc(2, 64, 8, 8, "NCHW"), F.bn_desc(2, 20, 8, 8), F.bn_desc(2, 24, 8, 8),
                F.bn_desc(2, 64, 8, 8, relu=False), F.bn_desc(2, 64, 8, 8, swap=True)):
        assert F.fp16_bn_mask_bytes(bad) == 0
    need = F.fp16_bn_workspace_bytes(d)
    M = Cc + (8 << 20)
    fw = [A, B, B + 256, Cc + (2 << 20), Cc, WS + (1 << 20), M, WS, need, None]
    assert lib.fp16_bn_relu_m(ctypes.byref(d), *fw[:6], None, *fw[7:]) == NULL
    assert lib.fp16_bn_relu_m(ctypes.byref(d), *fw[:6], M + 8, *fw[7:]) == MISALIGNED
    nc = F.bn_desc(2, 64, 8, 8, "NCHW")
    assert lib.fp16_bn_relu_m(ctypes.byref(nc), *fw) == UNSUPPORTED
    sw = F.bn_desc(2, 64, 8, 8, swap=True)
    assert lib.fp16_bn_relu_m(ctypes.byref(sw), *fw) == UNSUPPORTED
    for at in (A, Cc, Cc + (2 << 20), WS + (1 << 20), WS):  # x, y, residual, stats, workspace
        assert lib.fp16_bn_relu_m(ctypes.byref(d), *fw[:6], at, *fw[7:]) == ALIASING, hex(at)
    # backward: x, mask, dy, gamma, beta, stats, dx, dgamma, dbeta, dresidual, ws
    bw = [A, M, Cc, B, B + 256, WS + (1 << 20), Cc + (1 << 20), B + 512, B + 768, Cc + (3 << 20),
          WS, need, None]
    assert lib.fp16_bn_relu_bwd_m(ctypes.byref(d), bw[0], None, *bw[2:]) == NULL
    assert lib.fp16_bn_relu_bwd_m(ctypes.byref(nc), *bw) == UNSUPPORTED
    for i in (6, 9, 10):  # the mask under dx, dresidual or the workspace
        bad = list(bw)
        bad[i] = M
        assert lib.fp16_bn_relu_bwd_m(ctypes.byref(d), *bad) == ALIASING, i
    # the fused convolution + BN forward
    cd = _conv()
    bd = F.bn_desc(cd.n, cd.k, cd.h, cd.w)
    need = F.fp16_conv_bn_workspace_bytes(cd, bd)
    args = [A, B, B + (1 << 20), B + (1 << 20) + 256, None, Cc, Cc + (4 << 20), WS + (8 << 20)]
    assert lib.fp16_conv_bn_relu_fwd_m(ctypes.byref(cd), ctypes.byref(bd), *args, None, WS, need,
                                       None) == NULL
    assert lib.fp16_conv_bn_relu_fwd_m(ctypes.byref(cd), ctypes.byref(bd), *args, Cc + 64, WS,
                                       need, None) == ALIASING  # mask inside y
    assert lib.fp16_conv_bn_relu_fwd_m(ctypes.byref(cd), ctypes.byref(bd), *args, Cc + (4 << 20),
                                       WS, need, None) == ALIASING  # mask inside z


def test_bn_relu_maxpool_validation():
    lib = F.lib()
    f = lib.fp16_bn_relu_maxpool
    bd = F.bn_desc(2, 64, 112, 112)
    pd = F.pool_desc(2, 64, 112, 112, 3, 3, 2, 1)
    need = F.fp16_bn_workspace_bytes(bd)
    # x, gamma, beta, stats, y, idx, ws
    ok = [A, B, B + 256, B + 512, Cc, Cc + (8 << 20), WS, need, None]
    r = lambda b=bd, p=pd, args=ok: f(ctypes.byref(b), ctypes.byref(p), *args)
    assert f(None, ctypes.byref(pd), *ok) == NULL
    assert f(ctypes.byref(bd), None, *ok) == NULL
    for i in range(6):
        bad = list(ok)
        bad[i] = None
        assert r(args=bad) == NULL, i
    assert r(p=F.pool_desc(2, 64, 112, 110, 3, 3, 2, 1)) == SHAPE     # not the BN's tensor
    assert r(p=F.pool_desc(2, 64, 112, 112, 2, 2, 2, 0)) == UNSUPPORTED  # 2x2 window
    for b in (F.bn_desc(2, 64, 112, 112, relu=False), F.bn_desc(2, 64, 112, 112, swap=True),
              F.bn_desc(2, 24, 112, 112)):
        assert r(b=b, p=F.pool_desc(b.n, b.c, b.h, b.w, 3, 3, 2, 1)) == UNSUPPORTED
    nb, npd = F.bn_desc(2, 64, 112, 112, "NCHW"), F.pool_desc(2, 64, 112, 112, 3, 3, 2, 1, "NCHW")
    assert r(b=nb, p=npd) == UNSUPPORTED
    bad = list(ok)
    bad[4] = Cc + 8
    assert r(args=bad) == MISALIGNED
    assert r(args=ok[:6] + [WS, need - 16, None]) == WORKSPACE
    # y over x, idx over y, the workspace over stats
    for i, at in ((4, A + 64), (5, Cc + 64), (6, B)):
        bad = list(ok)
        bad[i] = at
        assert r(args=bad) == ALIASING, i


def test_dgrad_filters_validation():
    lib = F.lib()
    assert lib.fp16_conv_dgrad_filters(0, None, None, None, None) == OK  # nothing to do
    D = (F.ConvDesc * 2)(_conv(), _conv(k=128))
    P = lambda *a: (ctypes.c_void_p * len(a))(*a)
    assert lib.fp16_conv_dgrad_filters(-1, D, P(A), P(B), None) == SHAPE
    assert lib.fp16_conv_dgrad_filters(2, None, P(A, A + (1 << 20)), P(B, B + (1 << 20)), None) == NULL
    assert lib.fp16_conv_dgrad_filters(2, D, P(A, None), P(B, B + (1 << 20)), None) == NULL
    assert lib.fp16_conv_dgrad_filters(2, D, P(A, A + (1 << 20)), P(B, B + 8), None) == MISALIGNED
    # an output over another item's filter, or over another output
    assert lib.fp16_conv_dgrad_filters(2, D, P(A, A + (1 << 20)), P(B, A + (1 << 20) + 64),
                                       None) == ALIASING
    assert lib.fp16_conv_dgrad_filters(2, D, P(A, A + (1 << 20)), P(B, B + 256), None) == ALIASING
    N = (F.ConvDesc * 1)(_conv(layout="NCHW"))
    assert lib.fp16_conv_dgrad_filters(1, N, P(A), P(B), None) == UNSUPPORTED
    bad = (F.ConvDesc * 1)(_conv(n=0))
    assert lib.fp16_conv_dgrad_filters(1, bad, P(A), P(B), None) == SHAPE
