"""The bottleneck block's training step composed from the oracle's operations
-- TEST INFRASTRUCTURE ONLY (tests, smoke check, CPU-baseline timing).

Same block as the HIP path runs: 1x1 conv C->w, BN(0.25)+ReLU, 3x3 conv
w->w, BN(0.25)+ReLU, 1x1 conv w->C, BN(0.25) + identity shortcut + ReLU
(ResNet-50 bottleneck, Section 5.1; 0.25 multiplier, Section 4.2), then the
backward pass from a given output gradient and FP16 momentum SGD with weight
decay on the convolution weights only (Section 5.1).  Every stored tensor is
binary16 (Section 5.2); BN statistics are the oracle's own float64 ones.
Inputs are numpy arrays in NHWC / KRSC.
"""

from __future__ import annotations

import numpy as np

import oracle as O


def block_step(x, W, gamma, beta, dout, post_scale=0.25, eps=1e-5, lr=0.1, momentum=0.9,
               weight_decay=1e-4, mw=None, mbn=None):
    """One forward/backward/SGD step.  W: three KRSC filters; gamma/beta: three
    per-channel vectors.  Returns a dict of every stored tensor."""
    n, hw, _, c = x.shape
    shapes = [(w.shape[3], w.shape[0], w.shape[1]) for w in W]  # (C_in, C_out, R)
    cshp = [O.conv_shape(n, ci, hw, hw, co, r, r, 1, r // 2) for ci, co, r in shapes]
    bshp = [O.bn_shape(n, co, hw, hw) for _, co, _ in shapes]
    out = {}
    # forward
    inp = x
    cv, act = [], []
    for i in range(3):
        _, ci16 = O.conv_fwd(cshp[i], inp, W[i])
        res = x if i == 2 else None
        bn = O.bn_fwd(bshp[i], ci16, gamma[i], beta[i], res, eps, post_scale, True)
        cv.append(ci16)
        act.append(bn["y"])
        inp = bn["y"]
    # backward
    r3 = O.bn_bwd(bshp[2], cv[2], act[2], dout, gamma[2], eps, post_scale, True, want_dres=True)
    dcv = [None, None, r3["dx"]]
    dg = [None, None, r3["dgamma"]]
    db = [None, None, r3["dbeta"]]
    dW = [None, None, None]
    grad = r3["dx"]
    for i in (2, 1):
        _, dact = O.conv_dgrad(cshp[i], grad, W[i])
        _, dW[i] = O.conv_wgrad(cshp[i], act[i - 1], grad)
        r = O.bn_bwd(bshp[i - 1], cv[i - 1], act[i - 1], dact, gamma[i - 1], eps, post_scale, True)
        dcv[i - 1], dg[i - 1], db[i - 1] = r["dx"], r["dgamma"], r["dbeta"]
        grad = r["dx"]
    _, dx = O.conv_dgrad_add(cshp[0], grad, W[0], r3["dres"])
    _, dW[0] = O.conv_wgrad(cshp[0], x, grad)
    # SGD on the two parameter groups
    w_arena = np.concatenate([w.reshape(-1) for w in W])
    dw_arena = np.concatenate([g.reshape(-1) for g in dW])
    bn_arena = np.concatenate([v for pair in zip(gamma, beta) for v in pair])
    dbn_arena = np.concatenate([v for pair in zip(dg, db) for v in pair])
    mw = np.zeros_like(w_arena) if mw is None else mw
    mbn = np.zeros_like(bn_arena) if mbn is None else mbn
    w1, m1 = O.sgd_f32(w_arena, dw_arena, mw, lr, momentum, weight_decay)
    b1, mb1 = O.sgd_f32(bn_arena, dbn_arena, mbn, lr, momentum, 0.0)
    out.update(conv=cv, act=act, dconv=dcv, dW=dW, dgamma=dg, dbeta=db, dx=dx,
               dshort=r3["dres"], w_arena=w1, mw_arena=m1, bn_arena=b1, mbn_arena=mb1)
    return out


def block_flops(n, hw, shapes) -> int:
    """Convolution FLOPs of one pass over the block (2 per multiply-add)."""
    return sum(2 * n * hw * hw * co * ci * r * r for ci, co, r in shapes)
