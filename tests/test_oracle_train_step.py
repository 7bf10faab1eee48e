"""Pins for the oracle's composition of the whole ResNet-50 training step
(oracle/resnet50.py: forward, backward through every layer, SGD; the network
of Section 5.1 with the 0.25 multiplier of Section 4.2), built only from the
separately pinned oracle operations.  Its wiring is pinned by calculus:

- one SGD step along the composed gradient lowers the loss on the same batch
  (a wrong sign, a missing shortcut gradient or a dropped layer would not);
- the classifier bias gradient matches a central finite difference of the
  float64 batch loss in the bias (the loss is computed from binary16 logits,
  so the step is a multiple of their ulp).
"""

import numpy as np

import oracle
from oracle import resnet50 as net
from paper_1911_07384_amd import synth

STAGES = ((1, 8, 32, 1), (1, 16, 64, 2))


def _batch(n=4, hw=32, classes=10, seed=3):
    img = synth.normal_f16((n, hw, hw, 3), 1.0, seed, 1)
    lab = synth.labels(n, classes, seed, 2)
    return img, lab


def test_one_step_lowers_the_loss():
    img, lab = _batch()
    P = net.init_params(STAGES, classes=10, seed=4)
    loss0, G, P1, M1 = net.train_step(img, lab, P, lr=0.02, momentum=0.9, weight_decay=0.0,
                                      stages=STAGES)
    assert set(G) == set(P)
    for k, g in G.items():
        assert g.shape == P[k].shape and np.all(np.isfinite(g.astype(np.float32))), k
    loss1 = net.forward(img, lab, P1, stages=STAGES)[0]
    assert loss1 < loss0 - 1e-3, (loss0, loss1)
    # the momentum of the first step is the rounded gradient (zero-initialised buffer)
    for k in G:
        assert np.array_equal(M1[k].view(np.uint16), G[k].view(np.uint16)), k


def test_bias_gradient_matches_finite_difference():
    img, lab = _batch(seed=5)
    P = net.init_params(STAGES, classes=10, seed=6)
    _, G, _, _ = net.train_step(img, lab, P, lr=0.0, stages=STAGES)
    for j in (0, 3, 7):
        h = 2.0 ** -6
        Pp, Pm = dict(P), dict(P)
        bp, bm = P["fc.bias"].astype(np.float64).copy(), P["fc.bias"].astype(np.float64).copy()
        bp[j] += h
        bm[j] -= h
        Pp["fc.bias"], Pm["fc.bias"] = bp.astype(np.float16), bm.astype(np.float16)
        lp = net.forward(img, lab, Pp, stages=STAGES)[0]
        lm = net.forward(img, lab, Pm, stages=STAGES)[0]
        fd = (lp - lm) / (2 * h)
        assert abs(fd - float(G["fc.bias"][j])) <= 2e-2 * max(abs(fd), 1e-2), (j, fd, G["fc.bias"][j])
