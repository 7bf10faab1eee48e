"""ResNet-50's training step composed from the oracle's operations -- TEST
INFRASTRUCTURE ONLY (see this package's header).

The network of Section 5.1 of arXiv:1911.07384 (torchvision ResNet-50 v1.5):
7x7 stride-2 stem convolution, BN (no multiplier) and ReLU, 3x3 stride-2 max
pool, stages of 3, 4, 6, 3 bottlenecks (widths 64, 128, 256, 512, outputs 4x
the width, stride 2 on the 3x3 convolution of the first block of stages 2-4,
a 1x1 convolution + BN shortcut on each first block), global average pool,
2048 -> classes classifier with bias, softmax cross-entropy averaged over the
batch.  Every BN inside a residual block, the shortcut's included, is
followed by the 0.25 multiplier of Section 4.2.  Every tensor is stored in
binary16 between operations.

Parameters are passed in by name (``<stage>.<block>.<conv>`` for filters in
KRSC order, ``<bn name>.gamma`` / ``.beta``, ``fc`` and ``fc.bias``), so a test
can run the same weights through this composition and through the HIP path.
"""

from __future__ import annotations

import numpy as np

import oracle

STAGES = ((3, 64, 256, 1), (4, 128, 512, 2), (6, 256, 1024, 2), (3, 512, 2048, 2))


def _conv(x, w, stride, pad):
    n, h, wd, c = x.shape
    k, r, s, _ = w.shape
    shp = oracle.conv_shape(n, c, h, wd, k, r, s, stride, pad, "NHWC")
    return shp, oracle.conv_fwd(shp, x, w)[1]


def _bn(x, P, name, scale, relu, res=None, eps=1e-5):
    n, h, w, c = x.shape
    shp = oracle.bn_shape(n, c, h, w)
    out = oracle.bn_fwd(shp, x, P[name + ".gamma"], P[name + ".beta"], res, eps, scale, relu)
    return shp, out["y"]


def forward(image, labels, P, post_scale=0.25, stages=STAGES):
    """Returns (mean loss, per-sample losses, dict of every stored tensor)."""
    T = {}
    _, T["stem.y"] = _conv(image, P["stem"], 2, 3)
    _, T["stem.bn.y"] = _bn(T["stem.y"], P, "stem.bn", 1.0, True)
    n, h, w, c = T["stem.bn.y"].shape
    pshp = oracle.pool_shape(n, c, h, w, 3, 3, 2, 1, "NHWC")
    T["pool.y"], _ = oracle.maxpool_fwd(pshp, T["stem.bn.y"])
    x = T["pool.y"]
    for si, (nb, width, cout, stride) in enumerate(stages):
        for bi in range(nb):
            nm = f"l{si + 1}.{bi}"
            st = stride if bi == 0 else 1
            _, T[nm + ".c1.y"] = _conv(x, P[nm + ".c1"], 1, 0)
            _, T[nm + ".bn1.y"] = _bn(T[nm + ".c1.y"], P, nm + ".bn1", post_scale, True)
            _, T[nm + ".c2.y"] = _conv(T[nm + ".bn1.y"], P[nm + ".c2"], st, 1)
            _, T[nm + ".bn2.y"] = _bn(T[nm + ".c2.y"], P, nm + ".bn2", post_scale, True)
            _, T[nm + ".c3.y"] = _conv(T[nm + ".bn2.y"], P[nm + ".c3"], 1, 0)
            if bi == 0:
                _, T[nm + ".ds.y"] = _conv(x, P[nm + ".ds"], st, 0)
                _, T[nm + ".bnd.y"] = _bn(T[nm + ".ds.y"], P, nm + ".bnd", post_scale, False)
                res = T[nm + ".bnd.y"]
            else:
                res = x
            _, T[nm + ".bn3.y"] = _bn(T[nm + ".c3.y"], P, nm + ".bn3", post_scale, True, res)
            x = T[nm + ".bn3.y"]
    n, h, w, c = x.shape
    gshp = oracle.pool_shape(n, c, h, w, h, w, 1, 0, "NHWC")
    T["gap.y"] = oracle.avgpool_fwd(gshp, x)[1].reshape(n, 1, 1, c)
    _, T["fc.y"] = _conv(T["gap.y"], P["fc"], 1, 0)
    out = oracle.softmax_ce(T["fc.y"].reshape(n, -1), P["fc.bias"], labels)
    T["fc.dy"] = out["dz"].reshape(T["fc.y"].shape)
    T["fc.dbias"] = out["db"]
    return out["loss"], out["loss_rows"], T


def _bwd_bn(T, P, name, xname, dy, scale, relu, res=None, want_dres=False, eps=1e-5):
    x = T[xname]
    n, h, w, c = x.shape
    shp = oracle.bn_shape(n, c, h, w)
    return oracle.bn_bwd(shp, x, T[name + ".y"], dy, P[name + ".gamma"], eps, scale, relu,
                         want_dres=want_dres, residual=res)


def _bwd_conv(T, P, G, name, xname, dy, stride, pad, want_dx=True, addend=None):
    x, w = T[xname], P[name]
    n, h, wd, c = x.shape
    k, r, s, _ = w.shape
    shp = oracle.conv_shape(n, c, h, wd, k, r, s, stride, pad, "NHWC")
    G[name] = oracle.conv_wgrad(shp, x, dy)[1]
    if not want_dx:
        return None
    if addend is None:
        return oracle.conv_dgrad(shp, dy, w)[1]
    return oracle.conv_dgrad_add(shp, dy, w, addend)[1]


def train_step(image, labels, P, M=None, lr=0.1, momentum=0.9, weight_decay=1e-4,
               post_scale=0.25, stages=STAGES):
    """One whole training step: the forward above, the backward through every
    layer (the gradient of a block input is the branch's data gradient plus
    the shortcut's, rounded once), and momentum SGD on every parameter in
    binary16 (weight decay on filters, classifier weights and bias; none on
    BN parameters, Section 5.1).  M holds the momentum buffers by parameter
    name (zeros when absent).  Returns (mean loss, gradients, new parameters,
    new momenta)."""
    loss, _, T = forward(image, labels, P, post_scale, stages)
    G = {"fc.bias": T["fc.dbias"]}
    n = image.shape[0]
    dgap = _bwd_conv(T, P, G, "fc", "gap.y", T["fc.dy"], 1, 0)
    last = f"l{len(stages)}.{stages[-1][0] - 1}.bn3.y"
    x = T[last]
    gshp = oracle.pool_shape(n, x.shape[3], x.shape[1], x.shape[2], x.shape[1], x.shape[2], 1, 0,
                             "NHWC")
    dout = oracle.avgpool_bwd(gshp, dgap.reshape(n, -1))
    blocks = [(si, bi) for si, (nb, _, _, _) in enumerate(stages) for bi in range(nb)]
    for si, bi in reversed(blocks):
        nm = f"l{si + 1}.{bi}"
        st = stages[si][3] if bi == 0 else 1
        xin = "pool.y" if (si, bi) == (0, 0) else (f"l{si + 1}.{bi - 1}.bn3.y" if bi > 0 else
                                                   f"l{si}.{stages[si - 1][0] - 1}.bn3.y")
        res = T[nm + ".bnd.y"] if bi == 0 else T[xin]
        r3 = _bwd_bn(T, P, nm + ".bn3", nm + ".c3.y", dout, post_scale, True, res, True)
        G[nm + ".bn3.gamma"], G[nm + ".bn3.beta"] = r3["dgamma"], r3["dbeta"]
        d2 = _bwd_conv(T, P, G, nm + ".c3", nm + ".bn2.y", r3["dx"], 1, 0)
        r2 = _bwd_bn(T, P, nm + ".bn2", nm + ".c2.y", d2, post_scale, True)
        G[nm + ".bn2.gamma"], G[nm + ".bn2.beta"] = r2["dgamma"], r2["dbeta"]
        d1 = _bwd_conv(T, P, G, nm + ".c2", nm + ".bn1.y", r2["dx"], st, 1)
        r1 = _bwd_bn(T, P, nm + ".bn1", nm + ".c1.y", d1, post_scale, True)
        G[nm + ".bn1.gamma"], G[nm + ".bn1.beta"] = r1["dgamma"], r1["dbeta"]
        shortcut = r3["dres"]
        if bi == 0:
            rd = _bwd_bn(T, P, nm + ".bnd", nm + ".ds.y", shortcut, post_scale, False)
            G[nm + ".bnd.gamma"], G[nm + ".bnd.beta"] = rd["dgamma"], rd["dbeta"]
            shortcut = _bwd_conv(T, P, G, nm + ".ds", xin, rd["dx"], st, 0)
        dout = _bwd_conv(T, P, G, nm + ".c1", xin, r1["dx"], 1, 0, addend=shortcut)
    s = T["stem.bn.y"]
    pshp = oracle.pool_shape(n, s.shape[3], s.shape[1], s.shape[2], 3, 3, 2, 1, "NHWC")
    dstem = oracle.maxpool_bwd(pshp, s, dout)
    rs = _bwd_bn(T, P, "stem.bn", "stem.y", dstem, 1.0, True)
    G["stem.bn.gamma"], G["stem.bn.beta"] = rs["dgamma"], rs["dbeta"]
    T["image"] = image
    _bwd_conv(T, P, G, "stem", "image", rs["dx"], 2, 3, want_dx=False)
    newP, newM = {}, {}
    M = {} if M is None else M
    for name, g in G.items():
        w = P[name]
        m = M.get(name, np.zeros_like(w))
        wd = 0.0 if (".gamma" in name or ".beta" in name) else weight_decay
        w1, m1 = oracle.sgd_f32(w.reshape(-1), g.reshape(-1), m.reshape(-1), lr, momentum, wd)
        newP[name], newM[name] = w1.reshape(w.shape), m1.reshape(w.shape)
    return loss, G, newP, newM


def init_params(stages=STAGES, classes=1000, seed=0):
    """He-normal filters (KRSC, std sqrt(2 / fan_in)), gamma 1, beta 0, zero
    classifier bias, from the seeded generator shared with the HIP path."""
    from paper_1911_07384_amd import synth
    P, sid = {}, [1000]

    def filt(name, k, r, c):
        sid[0] += 1
        P[name] = synth.normal_f16((k, r, r, c), synth.he_std(c * r * r), seed, sid[0])

    def bn(name, c):
        P[name + ".gamma"] = np.ones(c, np.float16)
        P[name + ".beta"] = np.zeros(c, np.float16)

    filt("stem", 64, 7, 3)
    bn("stem.bn", 64)
    cin = 64
    for si, (nb, width, cout, _) in enumerate(stages):
        for bi in range(nb):
            nm = f"l{si + 1}.{bi}"
            filt(nm + ".c1", width, 1, cin)
            bn(nm + ".bn1", width)
            filt(nm + ".c2", width, 3, width)
            bn(nm + ".bn2", width)
            filt(nm + ".c3", cout, 1, width)
            bn(nm + ".bn3", cout)
            if bi == 0:
                filt(nm + ".ds", cout, 1, cin)
                bn(nm + ".bnd", cout)
            cin = cout
    filt("fc", classes, 1, cin)
    P["fc.bias"] = np.zeros(classes, np.float16)
    return P
