"""One ResNet-50 bottleneck block trained all in FP16 through the C ABI.

The block is torchvision's v1.5 bottleneck with an identity shortcut
(ResNet-50, Section 5.1 of arXiv:1911.07384): 1x1 conv C->w, 3x3 conv w->w,
1x1 conv w->C, each followed by BN with the 0.25 output multiplier of
Section 4.2 and ReLU, the last BN adding the shortcut before its ReLU.  One
training step is the forward pass, the backward pass from a given output
gradient, and FP16 momentum SGD on every parameter (weight decay on the
convolution weights, none on the BN parameters, Section 5.1).

Every tensor is binary16 in device memory (no master copy, Section 5.2); the
per-channel BN statistics are float32 buffers between forward and backward.
Parameters, gradients and momenta each live in one flat arena per
weight-decay group, so each SGD update is a single launch.  The weight
gradients are off the backward's critical path (nothing reads them before
the update), so they run on a second stream with their own workspace, each
after the BN backward that produces its input, and overlap the chain of
data gradients; the update waits for both streams.  Everything is enqueued
from the current stream (forked and joined with events), so a step can be
captured in a HIP graph.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

import paper_1911_07384_amd as F
from paper_1911_07384_amd import synth


@dataclass
class BlockShape:
    n: int = 32
    hw: int = 56
    c: int = 256      # block input/output channels
    width: int = 64   # bottleneck width
    post_scale: float = 0.25
    eps: float = 1e-5

    @property
    def conv_shapes(self):
        """(C_in, C_out, R) of the three convolutions."""
        return [(self.c, self.width, 1), (self.width, self.width, 3), (self.width, self.c, 1)]

    def conv_flops(self) -> int:
        """Algorithmic FLOPs of one pass (fwd, dgrad or wgrad) over the three convs."""
        m = self.n * self.hw * self.hw
        return sum(2 * m * co * ci * r * r for ci, co, r in self.conv_shapes)


class Bottleneck:
    """Device state and the ABI call sequence of one training step."""

    def __init__(self, shape: BlockShape = BlockShape(), seed: int = 0, device="cuda",
                 lr=0.1, momentum=0.9, weight_decay=1e-4, dy_std=1e-3, fuse_bn_stats=True):
        self.s = s = shape
        # each conv -> BN pair as one fused call (statistics in the conv epilogue)
        self.fuse = fuse_bn_stats
        self.lr, self.momentum, self.wd = lr, momentum, weight_decay
        n, hw, c, wdt = s.n, s.hw, s.c, s.width
        dev = torch.device(device)
        f16 = dict(dtype=torch.float16, device=dev)

        def put(a):
            return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

        # convolution weights (KRSC), He-normal with fan_in = C*R*S, in one arena
        self.conv_desc = []
        wsizes = []
        for (ci, co, r) in s.conv_shapes:
            self.conv_desc.append(F.conv_desc(n, ci, hw, hw, co, r, r, 1, r // 2))
            wsizes.append(co * r * r * ci)
        self.w_arena = torch.empty(sum(wsizes), **f16)
        self.dw_arena = torch.zeros(sum(wsizes), **f16)
        self.mw_arena = torch.zeros(sum(wsizes), **f16)
        self.W, self.dW = [], []
        off = 0
        for i, ((ci, co, r), sz) in enumerate(zip(s.conv_shapes, wsizes)):
            w = synth.normal_f16((co, r, r, ci), synth.he_std(ci * r * r), seed, 10 + i)
            self.w_arena[off:off + sz].copy_(put(w).reshape(-1))
            self.W.append(self.w_arena[off:off + sz].view(co, r, r, ci))
            self.dW.append(self.dw_arena[off:off + sz].view(co, r, r, ci))
            off += sz
        # BN parameters: gamma = 1, beta = 0, one arena [g1 b1 g2 b2 g3 b3]
        chans = [co for (_, co, _) in s.conv_shapes]
        self.bn_arena = torch.empty(2 * sum(chans), **f16)
        self.dbn_arena = torch.zeros_like(self.bn_arena)
        self.mbn_arena = torch.zeros_like(self.bn_arena)
        self.gamma, self.beta, self.dgamma, self.dbeta = [], [], [], []
        off = 0
        for co in chans:
            for lst, dlst, val in ((self.gamma, self.dgamma, 1.0), (self.beta, self.dbeta, 0.0)):
                self.bn_arena[off:off + co].fill_(val)
                lst.append(self.bn_arena[off:off + co])
                dlst.append(self.dbn_arena[off:off + co])
                off += co
        self.bn_desc = [F.bn_desc(n, co, hw, hw, "NHWC", s.eps, s.post_scale, True) for co in chans]
        self.stats = [torch.empty(2 * co, dtype=torch.float32, device=dev) for co in chans]

        # activations and gradients (NHWC)
        self.x = put(synth.normal_f16((n, hw, hw, c), 1.0, seed, 1))
        self.dout = put(synth.normal_f16((n, hw, hw, c), dy_std, seed, 2))
        self.cv = [torch.empty((n, hw, hw, co), **f16) for co in chans]   # conv outputs
        self.act = [torch.empty((n, hw, hw, co), **f16) for co in chans]  # BN/ReLU outputs
        self.dcv = [torch.empty((n, hw, hw, co), **f16) for co in chans]  # grads at conv outputs
        self.dact = [torch.empty((n, hw, hw, co), **f16) for co in chans[:2]]  # grads at a1, a2
        self.dshort = torch.empty((n, hw, hw, c), **f16)  # gradient through the shortcut
        self.dx = torch.empty((n, hw, hw, c), **f16)

        # one workspace shared by every call (they run in order on one stream)
        need = 0
        for d in self.conv_desc:
            for p in (F.PASS_FWD, F.PASS_DGRAD, F.PASS_WGRAD):
                need = max(need, F.fp16_conv_workspace_bytes(d, p))
        for d in self.bn_desc:
            need = max(need, F.fp16_bn_workspace_bytes(d))
        for cd, bd in zip(self.conv_desc, self.bn_desc):
            need = max(need, F.fp16_conv_bn_workspace_bytes(cd, bd))
        self.ws = F.workspace(need, dev)
        self.ws_side = F.workspace(need, dev)  # the weight-gradient stream's own workspace
        self.side = torch.cuda.Stream(device=dev) if dev.type == "cuda" else None

    # ---- the step, one ABI call per line -------------------------------------

    def forward(self):
        d, ws = self.conv_desc, self.ws
        if self.fuse:
            ins, res = [self.x, self.act[0], self.act[1]], [None, None, self.x]
            for i in range(3):
                F.fp16_conv_bn_relu_fwd(d[i], self.bn_desc[i], ins[i], self.W[i], self.gamma[i],
                                        self.beta[i], res[i], self.cv[i], self.act[i],
                                        self.stats[i], ws)
            return
        F.fp16_conv_fwd(d[0], self.x, self.W[0], self.cv[0], ws)
        F.fp16_bn_relu(self.bn_desc[0], self.cv[0], self.gamma[0], self.beta[0], None, self.act[0],
                       self.stats[0], ws)
        F.fp16_conv_fwd(d[1], self.act[0], self.W[1], self.cv[1], ws)
        F.fp16_bn_relu(self.bn_desc[1], self.cv[1], self.gamma[1], self.beta[1], None, self.act[1],
                       self.stats[1], ws)
        F.fp16_conv_fwd(d[2], self.act[1], self.W[2], self.cv[2], ws)
        F.fp16_bn_relu(self.bn_desc[2], self.cv[2], self.gamma[2], self.beta[2], self.x, self.act[2],
                       self.stats[2], ws)

    def backward(self):
        d, ws, wss = self.conv_desc, self.ws, self.ws_side
        main, side = torch.cuda.current_stream(), self.side

        def wgrad_after(i, x, dy):
            # the weight gradient of conv i on the side stream, once dy exists
            ev = torch.cuda.Event()
            ev.record(main)
            side.wait_event(ev)
            with torch.cuda.stream(side):
                F.fp16_conv_wgrad(d[i], x, dy, self.dW[i], wss)

        # ReLU masks are recomputed from the conv outputs and statistics (y = None)
        F.fp16_bn_relu_bwd(self.bn_desc[2], self.cv[2], None, self.dout, self.gamma[2], self.beta[2],
                           self.x, self.stats[2], self.dcv[2], self.dgamma[2], self.dbeta[2],
                           self.dshort, ws)
        wgrad_after(2, self.act[1], self.dcv[2])
        F.fp16_conv_dgrad(d[2], self.dcv[2], self.W[2], self.dact[1], ws)
        F.fp16_bn_relu_bwd(self.bn_desc[1], self.cv[1], None, self.dact[1], self.gamma[1],
                           self.beta[1], None, self.stats[1], self.dcv[1], self.dgamma[1],
                           self.dbeta[1], None, ws)
        wgrad_after(1, self.act[0], self.dcv[1])
        F.fp16_conv_dgrad(d[1], self.dcv[1], self.W[1], self.dact[0], ws)
        F.fp16_bn_relu_bwd(self.bn_desc[0], self.cv[0], None, self.dact[0], self.gamma[0],
                           self.beta[0], None, self.stats[0], self.dcv[0], self.dgamma[0],
                           self.dbeta[0], None, ws)
        wgrad_after(0, self.x, self.dcv[0])
        F.fp16_conv_dgrad_add(d[0], self.dcv[0], self.W[0], self.dshort, self.dx, ws)
        main.wait_stream(side)  # the update reads every weight gradient

    def update(self):
        F.fp16_sgd_step(self.w_arena, self.dw_arena, self.mw_arena, self.w_arena.numel(), self.lr,
                        self.momentum, self.wd)
        F.fp16_sgd_step(self.bn_arena, self.dbn_arena, self.mbn_arena, self.bn_arena.numel(),
                        self.lr, self.momentum, 0.0)

    def step(self):
        self.forward()
        self.backward()
        self.update()

    # ---- the same calls, named, for per-call timing --------------------------

    def calls(self):
        """(name, thunk) for every ABI call of one step, in order."""
        d, ws, bd = self.conv_desc, self.ws, self.bn_desc
        c = []
        if self.fuse:
            ins, res = [self.x, self.act[0], self.act[1]], [None, None, self.x]
            for i in range(3):
                c.append((f"conv{i + 1}_bn{i + 1}_fwd",
                          lambda i=i: F.fp16_conv_bn_relu_fwd(d[i], bd[i], ins[i], self.W[i],
                                                              self.gamma[i], self.beta[i], res[i],
                                                              self.cv[i], self.act[i],
                                                              self.stats[i], ws)))
        else:
            c.append(("conv1_fwd", lambda: F.fp16_conv_fwd(d[0], self.x, self.W[0], self.cv[0], ws)))
            c.append(("bn1_fwd", lambda: F.fp16_bn_relu(bd[0], self.cv[0], self.gamma[0], self.beta[0],
                                                        None, self.act[0], self.stats[0], ws)))
            c.append(("conv2_fwd", lambda: F.fp16_conv_fwd(d[1], self.act[0], self.W[1], self.cv[1], ws)))
            c.append(("bn2_fwd", lambda: F.fp16_bn_relu(bd[1], self.cv[1], self.gamma[1], self.beta[1],
                                                        None, self.act[1], self.stats[1], ws)))
            c.append(("conv3_fwd", lambda: F.fp16_conv_fwd(d[2], self.act[1], self.W[2], self.cv[2], ws)))
            c.append(("bn3_fwd", lambda: F.fp16_bn_relu(bd[2], self.cv[2], self.gamma[2], self.beta[2],
                                                        self.x, self.act[2], self.stats[2], ws)))
        c.append(("bn3_bwd", lambda: F.fp16_bn_relu_bwd(
            bd[2], self.cv[2], None, self.dout, self.gamma[2], self.beta[2], self.x, self.stats[2],
            self.dcv[2], self.dgamma[2], self.dbeta[2], self.dshort, ws)))
        c.append(("conv3_dgrad", lambda: F.fp16_conv_dgrad(d[2], self.dcv[2], self.W[2],
                                                           self.dact[1], ws)))
        c.append(("conv3_wgrad", lambda: F.fp16_conv_wgrad(d[2], self.act[1], self.dcv[2],
                                                           self.dW[2], ws)))
        c.append(("bn2_bwd", lambda: F.fp16_bn_relu_bwd(
            bd[1], self.cv[1], None, self.dact[1], self.gamma[1], self.beta[1], None, self.stats[1],
            self.dcv[1], self.dgamma[1], self.dbeta[1], None, ws)))
        c.append(("conv2_dgrad", lambda: F.fp16_conv_dgrad(d[1], self.dcv[1], self.W[1],
                                                           self.dact[0], ws)))
        c.append(("conv2_wgrad", lambda: F.fp16_conv_wgrad(d[1], self.act[0], self.dcv[1],
                                                           self.dW[1], ws)))
        c.append(("bn1_bwd", lambda: F.fp16_bn_relu_bwd(
            bd[0], self.cv[0], None, self.dact[0], self.gamma[0], self.beta[0], None, self.stats[0],
            self.dcv[0], self.dgamma[0], self.dbeta[0], None, ws)))
        c.append(("conv1_dgrad_add", lambda: F.fp16_conv_dgrad_add(d[0], self.dcv[0], self.W[0],
                                                                   self.dshort, self.dx, ws)))
        c.append(("conv1_wgrad", lambda: F.fp16_conv_wgrad(d[0], self.x, self.dcv[0], self.dW[0],
                                                           ws)))
        c.append(("sgd_conv", lambda: F.fp16_sgd_step(self.w_arena, self.dw_arena, self.mw_arena,
                                                      self.w_arena.numel(), self.lr, self.momentum,
                                                      self.wd)))
        c.append(("sgd_bn", lambda: F.fp16_sgd_step(self.bn_arena, self.dbn_arena, self.mbn_arena,
                                                    self.bn_arena.numel(), self.lr, self.momentum,
                                                    0.0)))
        return c

    # ---- state snapshots (for graph-vs-eager checks and restarts) ------------

    def state(self):
        return [t.clone() for t in (self.w_arena, self.mw_arena, self.bn_arena, self.mbn_arena)]

    def load_state(self, st):
        for t, v in zip((self.w_arena, self.mw_arena, self.bn_arena, self.mbn_arena), st):
            t.copy_(v)
