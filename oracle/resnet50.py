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
