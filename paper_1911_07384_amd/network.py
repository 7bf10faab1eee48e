"""ResNet-50 trained all in FP16 through the C ABI: one training step of the
whole network on one GPU's batch (Section 5.1 of arXiv:1911.07384).

The network is torchvision's ResNet-50 v1.5 (stride on the 3x3 convolution
of each downsampling bottleneck): a 7x7 stride-2 stem convolution with BN and
ReLU, a 3x3 stride-2 max pool, four stages of 3, 4, 6 and 3 bottleneck
blocks, global average pooling and a 2048->1000 classifier with bias,
trained with the softmax cross-entropy averaged over the batch.  Every BN
inside a residual block is followed by the 0.25 multiplier (Section 4.2),
including the BN of a downsampling shortcut; the stem BN is not.  All
tensors are binary16 (no master copy, no loss scaling, Section 5.2); the SGD
step runs over two flat parameter arenas (weight decay on the convolution
and classifier weights and the classifier bias, none on BN parameters,
Section 5.1).

Options: ``bn_swap`` makes every block-last BN the BN swap of Section 4.1
(the shortcut joins before gamma); ``zero_gamma_last`` starts every
block-last gamma at 0 (the initialisation of Section 5.1; with the swap it
also zeroes the shortcut's contribution at the start).

The step is an explicit program: a list of ``Op`` records, each one ABI call
with named device buffers.  Running the list in order is one training step.
A downsampling block's shortcut convolution + BN runs on a second stream
beside the block's first two convolutions in the forward.  The weight
gradients are off the backward's critical path, so ``backward``
runs them on a second stream with their own workspace, each after an event
from the call that produced its input gradient, and joins the streams before
the update; everything else runs in order on the current stream.  The step
can be captured in a HIP graph.  The records also let tests replay any
call's inputs through the oracle.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

import paper_1911_07384_amd as F
from paper_1911_07384_amd import synth

STAGES = ((3, 64, 256, 1), (4, 128, 512, 2), (6, 256, 1024, 2), (3, 512, 2048, 2))


@dataclass
class Op:
    kind: str
    name: str
    a: dict = field(default_factory=dict)


class ResNet50:
    """Device state and the ABI program of one ResNet-50 training step."""

    # split-K workgroups of a weight gradient on the second stream, by stage
    # (the classifier's: the last entry): at batch 128 the step took 12.49 ms
    # with the default 512 (two per CU) everywhere, 12.20 with 256, 12.22 with
    # 224 and 12.37 with 320 (fewer float32 partial sums, more of the device
    # left to the memory-bound calls beside them; 128 and 64 made the weight
    # gradients the critical path); then 192 for stage 1 and 224 for stage 2
    # took another 0.07 ms
    SIDE_WORKGROUPS = (192, 224, 256, 256, 256)

    def __init__(self, n: int = 128, image: int = 224, classes: int = 1000, seed: int = 0,
                 lr: float = 0.1, momentum: float = 0.9, weight_decay: float = 1e-4,
                 post_scale: float = 0.25, eps: float = 1e-5, stages=STAGES, device="cuda",
                 bn_swap: bool = False, zero_gamma_last: bool = False,
                 fuse_bn_stats: bool = True):
        self.n, self.image, self.classes = n, image, classes
        self.lr, self.momentum, self.wd = lr, momentum, weight_decay
        self.post_scale, self.eps = post_scale, eps
        self.bn_swap, self.zero_gamma_last = bn_swap, zero_gamma_last
        self.fuse = fuse_bn_stats
        self.seed = seed
        self.dev = torch.device(device)
        self._stream_id = 100
        self.convs = []    # (name, desc, W view, dW view)
        self.bns = []      # (name, channels)
        self._wspecs = []  # (name, shape, std) of every weight-decay parameter
        self._bnspecs = []
        self.fwd, self.bwd, self.upd = [], [], []
        self.prep = []     # data-gradient filter rearrangements, run during the forward
        self.buffers = {}
        self._ws_need = 0
        self._plan(stages)
        self._allocate_params()
        self.ws = F.workspace(self._ws_need, self.dev)
        self.ws_side = F.workspace(self._ws_need, self.dev)  # the weight-gradient stream's
        self.side = torch.cuda.Stream(device=self.dev) if self.dev.type == "cuda" else None
        self._schedule()

    # ---- buffers -------------------------------------------------------------

    def _buf(self, name, shape, dtype=torch.float16):
        t = torch.empty(shape, dtype=dtype, device=self.dev)
        self.buffers[name] = t
        return t

    def _next_stream(self):
        self._stream_id += 1
        return self._stream_id

    # ---- planning: shapes, buffers and the op lists -------------------------------

    def _conv(self, name, x, xname, ci, co, r, stride, pad):
        n, h = x.shape[0], x.shape[1]
        d = F.conv_desc(n, ci, h, h, co, r, r, stride, pad)
        p, q = F.fp16_conv_out_dims(d)
        for ps in (F.PASS_FWD, F.PASS_DGRAD, F.PASS_WGRAD):
            self._ws_need = max(self._ws_need, F.fp16_conv_workspace_bytes(d, ps))
        y = self._buf(name + ".y", (n, p, q, co))
        self._wspecs.append((name, (co, r, r, ci), synth.he_std(ci * r * r)))
        self.convs.append({"name": name, "desc": d, "x": xname, "y": name + ".y"})
        self.fwd.append(Op("conv_fwd", name, {"desc": d, "x": xname, "w": name, "y": name + ".y"}))
        return y

    def _bn(self, name, x, xname, relu, post_scale, res=None, swap=False):
        n, h, w, c = x.shape
        d = F.bn_desc(n, c, h, w, "NHWC", self.eps, post_scale, relu, swap=swap)
        self._ws_need = max(self._ws_need, F.fp16_bn_workspace_bytes(d))
        y = self._buf(name + ".y", x.shape)
        self._buf(name + ".stats", (2 * c,), torch.float32)
        self._bnspecs.append((name, c))
        a = {"desc": d, "x": xname, "res": res, "y": name + ".y", "stats": name + ".stats",
             "mask": None}
        # a BN whose ReLU follows the shortcut keeps its ReLU mask for the
        # backward (one bit per element instead of reading the shortcut again)
        mb = F.fp16_bn_mask_bytes(d) if (res is not None and relu and not swap) else 0
        if mb:
            self._buf(name + ".mask", (mb,), torch.uint8)
            a["mask"] = name + ".mask"
        self.fwd.append(Op("bn_fwd", name, a))
        return y

    def _plan(self, stages):
        n, s = self.n, self.post_scale
        img = self._buf("image", (n, self.image, self.image, 3))
        self._buf("labels", (n,), torch.int32)
        # stem: conv 7x7/2, BN (multiplier 1) + ReLU, max pool 3x3/2
        y = self._conv("stem", img, "image", 3, 64, 7, 2, 3)
        a = self._bn("stem.bn", y, "stem.y", True, 1.0)
        pd = F.pool_desc(n, 64, a.shape[1], a.shape[2], 3, 3, 2, 1)
        p, q = F.fp16_pool_out_dims(pd)
        self._buf("pool.y", (n, p, q, 64))
        self._buf("pool.idx", (n, p, q, 64), torch.uint8)
        self.fwd.append(Op("maxpool_fwd", "pool", {"desc": pd, "x": "stem.bn.y", "y": "pool.y",
                                                   "idx": "pool.idx"}))
        x, xname, cin = self.buffers["pool.y"], "pool.y", 64
        self.blocks = []
        for si, (nb, width, cout, stride) in enumerate(stages):
            for bi in range(nb):
                nm = f"l{si + 1}.{bi}"
                st = stride if bi == 0 else 1
                blk = {"name": nm, "x": xname, "ds": bi == 0}
                y1 = self._conv(nm + ".c1", x, xname, cin, width, 1, 1, 0)
                a1 = self._bn(nm + ".bn1", y1, nm + ".c1.y", True, s)
                y2 = self._conv(nm + ".c2", a1, nm + ".bn1.y", width, width, 3, st, 1)
                a2 = self._bn(nm + ".bn2", y2, nm + ".c2.y", True, s)
                if bi == 0:  # the shortcut first, so that c3 is followed by its BN
                    yd = self._conv(nm + ".ds", x, xname, cin, cout, 1, st, 0)
                    self._bn(nm + ".bnd", yd, nm + ".ds.y", False, s)
                    res = nm + ".bnd.y"
                else:
                    res = xname
                y3 = self._conv(nm + ".c3", a2, nm + ".bn2.y", width, cout, 1, 1, 0)
                blk["res"] = res
                out = self._bn(nm + ".bn3", y3, nm + ".c3.y", True, s, res=res,
                               swap=self.bn_swap)
                self.blocks.append(blk)
                x, xname, cin = out, nm + ".bn3.y", cout
        # global average pool to [N, 1, 1, C], classifier as a 1x1 convolution
        h = x.shape[1]
        gd = F.pool_desc(n, cin, h, h, h, h, 1, 0)
        self._buf("gap.y", (n, 1, 1, cin))
        self.fwd.append(Op("avgpool_fwd", "gap", {"desc": gd, "x": xname, "y": "gap.y"}))
        self._conv("fc", self.buffers["gap.y"], "gap.y", cin, self.classes, 1, 1, 0)
        self._buf("loss", (n,), torch.float32)
        self._buf("fc.dy", (n, 1, 1, self.classes))
        self.fwd.append(Op("softmax_ce", "loss", {"n": n, "k": self.classes, "z": "fc.y",
                                                  "bias": "fc.bias", "labels": "labels",
                                                  "loss": "loss", "dz": "fc.dy",
                                                  "dbias": "fc.dbias"}))
        self._last = xname
        self._plan_backward(gd, pd)
        if self.fuse:
            self._fuse_bn_pool()
            self._fuse_conv_bn()

    def _fuse_bn_pool(self):
        """A BN + ReLU whose output only feeds the max pool that follows it
        (the stem's) becomes one fp16_bn_relu_maxpool call: the BN output is
        never written (its backward recomputes the ReLU mask from the BN input
        and the statistics), so its buffer is dropped."""
        out, i = [], 0
        while i < len(self.fwd):
            op = self.fwd[i]
            nxt = self.fwd[i + 1] if i + 1 < len(self.fwd) else None
            if (op.kind == "bn_fwd" and nxt is not None and nxt.kind == "maxpool_fwd"
                    and nxt.a["x"] == op.a["y"] and op.a["res"] is None and op.a["mask"] is None
                    and op.a["desc"].relu and not self._reads_elsewhere(op.a["y"], nxt)):
                out.append(Op("bn_maxpool_fwd", op.name,
                              {"desc": op.a["desc"], "pool": nxt.a["desc"], "x": op.a["x"],
                               "stats": op.a["stats"], "y": nxt.a["y"], "idx": nxt.a["idx"]}))
                del self.buffers[op.a["y"]]
                i += 2
            else:
                out.append(op)
                i += 1
        self.fwd = out

    def _reads_elsewhere(self, buf, but):
        """Whether any call of the step other than `but` reads buffer `buf`."""
        for op in self.fwd + self.bwd:
            if op is not but and any(isinstance(v, str) and v == buf and
                                     k not in self._OUTPUTS[op.kind] for k, v in op.a.items()):
                return True
        return False

    def _fuse_conv_bn(self):
        """Each conv whose next forward call is the BN of its output becomes
        one fp16_conv_bn_relu_fwd call (statistics in the conv epilogue)."""
        out, i = [], 0
        while i < len(self.fwd):
            op = self.fwd[i]
            nxt = self.fwd[i + 1] if i + 1 < len(self.fwd) else None
            if (op.kind == "conv_fwd" and nxt is not None and nxt.kind == "bn_fwd"
                    and nxt.a["x"] == op.a["y"] and op.a["desc"].k % 8 == 0):
                self._ws_need = max(self._ws_need,
                                    F.fp16_conv_bn_workspace_bytes(op.a["desc"], nxt.a["desc"]))
                out.append(Op("conv_bn_fwd", nxt.name,
                              {"desc": op.a["desc"], "bn": nxt.a["desc"], "x": op.a["x"],
                               "w": op.a["w"], "y": op.a["y"], "z": nxt.a["y"],
                               "res": nxt.a["res"], "stats": nxt.a["stats"],
                               "mask": nxt.a["mask"], "conv": op.name}))
                i += 2
            else:
                out.append(op)
                i += 1
        self.fwd = out

    def _grad(self, name):
        """Gradient buffer shaped like buffer `name`, registered as d:<name>."""
        key = "d:" + name
        if key not in self.buffers:
            src = self.buffers[name]
            self.buffers[key] = torch.empty(src.shape, dtype=src.dtype, device=self.dev)
        return key

    def _conv_op(self, name):
        return next(c for c in self.convs if c["name"] == name)

    def _bn_op(self, name):
        return next(o for o in self.fwd if o.kind == "bn_fwd" and o.name == name)

    def _bn_bwd(self, name, dy, want_dres, mask_of=None):
        """The backward of BN `name`; with mask_of, dy is the gradient the BN
        mask_of received and this BN's output reached mask_of's ReLU through
        the shortcut, so its incoming gradient is dy under mask_of's kept mask
        (the call is the ReLU form with that mask)."""
        f = self._bn_op(name).a
        dx = self._grad(f["x"])
        desc, mask = f["desc"], f["mask"]
        if mask_of is not None:
            d = desc
            desc = F.bn_desc(d.n, d.c, d.h, d.w, "NHWC", d.eps, d.post_scale, True)
            mask = self._bn_op(mask_of).a["mask"]
        a = {"desc": desc, "x": f["x"], "y": None, "dy": dy, "res": f["res"],
             "stats": f["stats"], "dx": dx, "dgamma": name + ".dgamma", "dbeta": name + ".dbeta",
             "dres": None, "mask": mask, "mask_of": mask_of or name}
        if want_dres:
            a["dres"] = self._grad(f["res"]) if f["res"] is not None else None
        self.bwd.append(Op("bn_bwd", name, a))
        return dx

    def _conv_bwd(self, name, dy, dx_needed=True, addend=None, dx_name=None, mask_of=None,
                  dgrad_desc=None, addend_stride=1):
        """The data gradient (with dgrad_desc: computed as that problem instead,
        e.g. a strided 1x1 convolution's on its own output grid) and the weight
        gradient of convolution `name`."""
        c = self._conv_op(name)
        if dx_needed:
            dx = dx_name or self._grad(c["x"])
            dd = dgrad_desc or c["desc"]
            # the filter is rearranged for the data gradient during the forward
            # (on the side stream, off the critical path); the data gradient
            # reads the rearranged copy
            wf = name + ".wf"
            self._buf(wf, (F.fp16_conv_dgrad_filter_bytes(dd) // 2,))
            self.prep.append(Op("dgrad_filter", name, {"desc": dd, "w": name, "wf": wf}))
            if addend is None:
                self.bwd.append(Op("conv_dgrad", name, {"desc": dd, "dy": dy, "w": name,
                                                        "wf": wf, "dx": dx}))
            else:
                # with mask_of, the addend is the gradient the BN mask_of
                # received, taken under that BN's kept ReLU mask; with
                # addend_stride s, it holds every s-th row and column only
                self.bwd.append(Op("conv_dgrad_add", name, {
                    "desc": dd, "dy": dy, "w": name, "wf": wf, "addend": addend,
                    "amask": self._bn_op(mask_of).a["mask"] if mask_of else None,
                    "mask_of": mask_of, "astride": addend_stride, "dx": dx}))
        # the weight gradients beside the backward's other calls aim at about
        # one workgroup per CU; the first layer's, the last call of the
        # backward with nothing left to overlap, takes the default two
        stage = int(name[1]) - 1 if name[0] == "l" else -1
        wg = self.SIDE_WORKGROUPS[stage] if dx_needed else 0
        self.bwd.append(Op("conv_wgrad", name, {"desc": c["desc"], "x": c["x"], "dy": dy,
                                                "dw": "d:" + name, "wg": wg}))

    def _plan_backward(self, gd, pd):
        # classifier: the loss kernel wrote fc.dy and the bias gradient
        self._conv_bwd("fc", "fc.dy")
        dgap = self._grad("gap.y")
        dlast = self._grad(self._last)
        self.bwd.append(Op("avgpool_bwd", "gap", {"desc": gd, "dy": dgap, "dx": dlast}))
        dout = dlast
        for blk in reversed(self.blocks):
            nm = blk["name"]
            # a block-last BN that kept its ReLU mask writes no shortcut
            # gradient: it is that BN's incoming gradient under the mask, and
            # its readers (the block input's data gradient, or the shortcut
            # BN's backward) take it that way
            kept = self._bn_op(nm + ".bn3").a["mask"] is not None
            dc3 = self._bn_bwd(nm + ".bn3", dout, want_dres=not kept)
            dres = "d:" + self._bn_op(nm + ".bn3").a["res"]
            self._conv_bwd(nm + ".c3", dc3)
            dc2 = self._bn_bwd(nm + ".bn2", "d:" + nm + ".bn2.y", want_dres=False)
            self._conv_bwd(nm + ".c2", dc2)
            dc1 = self._bn_bwd(nm + ".bn1", "d:" + nm + ".bn1.y", want_dres=False)
            # block input gradient = branch gradient + shortcut gradient, one rounding
            dxb = "dx:" + nm
            self.buffers[dxb] = torch.empty(self.buffers[blk["x"]].shape, dtype=torch.float16,
                                            device=self.dev)
            if blk["ds"]:
                if kept:
                    dcd = self._bn_bwd(nm + ".bnd", dout, want_dres=False, mask_of=nm + ".bn3")
                else:
                    dcd = self._bn_bwd(nm + ".bnd", dres, want_dres=False)
                dsx = "dds:" + nm
                d = self._conv_op(nm + ".ds")["desc"]
                if d.stride_h > 1:
                    # a strided 1x1 shortcut's data gradient is nonzero on its
                    # own grid only: computed there (a 1x1 stride-1 problem)
                    # and added by the block input's data gradient as a
                    # strided addend, instead of written out three zeros in four
                    p, q = F.fp16_conv_out_dims(d)
                    dc = F.conv_desc(d.n, d.c, p, q, d.k, 1, 1, 1, 0)
                    self.buffers[dsx] = torch.empty((d.n, p, q, d.c), dtype=torch.float16,
                                                    device=self.dev)
                    self._ws_need = max(self._ws_need, F.fp16_conv_workspace_bytes(dc, F.PASS_DGRAD))
                    self._conv_bwd(nm + ".ds", dcd, dx_name=dsx, dgrad_desc=dc)
                    self._conv_bwd(nm + ".c1", dc1, addend=dsx, dx_name=dxb,
                                   addend_stride=d.stride_h)
                else:
                    self.buffers[dsx] = torch.empty_like(self.buffers[dxb])
                    self._conv_bwd(nm + ".ds", dcd, dx_name=dsx)
                    self._conv_bwd(nm + ".c1", dc1, addend=dsx, dx_name=dxb)
            elif kept:
                self._conv_bwd(nm + ".c1", dc1, addend=dout, dx_name=dxb, mask_of=nm + ".bn3")
            else:
                self._conv_bwd(nm + ".c1", dc1, addend=dres, dx_name=dxb)
            dout = dxb
        # max pool, stem BN (its ReLU mask recomputed from the conv output and
        # the statistics, as for every other BN: reading the stored output
        # instead would add 2 bytes per element to both backward passes), stem
        # weights (the image gradient is not needed)
        dstem = self._grad("stem.bn.y")
        self.bwd.append(Op("maxpool_bwd", "pool", {"desc": pd, "idx": "pool.idx", "dy": dout,
                                                   "dx": dstem}))
        dc = self._bn_bwd("stem.bn", dstem, want_dres=False)
        self._conv_bwd("stem", dc, dx_needed=False)

    # ---- parameters ----------------------------------------------------------------

    def _allocate_params(self):
        f16 = dict(dtype=torch.float16, device=self.dev)
        sizes = [int(np.prod(sh)) for _, sh, _ in self._wspecs]
        nw = sum(sizes) + self.classes  # + classifier bias
        self.w_arena = torch.empty(nw, **f16)
        self.dw_arena = torch.zeros(nw, **f16)
        self.mw_arena = torch.zeros(nw, **f16)
        off = 0
        for (name, sh, std), sz in zip(self._wspecs, sizes):
            w = synth.normal_f16(sh, std, self.seed, self._next_stream())
            self.w_arena[off:off + sz].copy_(torch.from_numpy(w.reshape(-1)).to(self.dev))
            self.buffers[name] = self.w_arena[off:off + sz].view(sh)
            self.buffers["d:" + name] = self.dw_arena[off:off + sz].view(sh)
            off += sz
        self.w_arena[off:].zero_()
        self.buffers["fc.bias"] = self.w_arena[off:]
        self.buffers["fc.dbias"] = self.dw_arena[off:]
        nb = 2 * sum(c for _, c in self._bnspecs)
        self.bn_arena = torch.empty(nb, **f16)
        self.dbn_arena = torch.zeros(nb, **f16)
        self.mbn_arena = torch.zeros(nb, **f16)
        off = 0
        for name, c in self._bnspecs:
            last = name.endswith(".bn3") and self.zero_gamma_last
            self.bn_arena[off:off + c].fill_(0.0 if last else 1.0)
            self.buffers[name + ".gamma"] = self.bn_arena[off:off + c]
            self.buffers[name + ".dgamma"] = self.dbn_arena[off:off + c]
            off += c
            self.bn_arena[off:off + c].fill_(0.0)
            self.buffers[name + ".beta"] = self.bn_arena[off:off + c]
            self.buffers[name + ".dbeta"] = self.dbn_arena[off:off + c]
            off += c
        self.upd = [
            Op("sgd", "sgd_weights", {"w": self.w_arena, "g": self.dw_arena, "m": self.mw_arena,
                                      "wd": self.wd}),
            Op("sgd", "sgd_bn", {"w": self.bn_arena, "g": self.dbn_arena, "m": self.mbn_arena,
                                 "wd": 0.0}),
        ]
        self.n_weights, self.n_bn = nw, nb

    def load_batch(self, seed: int = 0):
        """Synthetic images ~ N(0, 1) and uniform labels (the ImageNet shapes)."""
        img = synth.normal_f16((self.n, self.image, self.image, 3), 1.0, seed, 1)
        lab = synth.labels(self.n, self.classes, seed, 2)
        self.buffers["image"].copy_(torch.from_numpy(img).to(self.dev))
        self.buffers["labels"].copy_(torch.from_numpy(lab).to(self.dev))

    # ---- execution -------------------------------------------------------------------

    def _t(self, key):
        return None if key is None else self.buffers[key]

    def run(self, op: Op, ws=None) -> None:
        a, t = op.a, self._t
        ws = self.ws if ws is None else ws
        k = op.kind
        if k == "conv_fwd":
            F.fp16_conv_fwd(a["desc"], t(a["x"]), t(a["w"]), t(a["y"]), ws)
        elif k == "conv_dgrad":
            F.fp16_conv_dgrad_wf(a["desc"], t(a["dy"]), t(a["wf"]), None, t(a["dx"]), ws)
        elif k == "conv_dgrad_add":
            if a["amask"] is None and a["astride"] == 1:
                F.fp16_conv_dgrad_wf(a["desc"], t(a["dy"]), t(a["wf"]), t(a["addend"]), t(a["dx"]),
                                     ws)
            elif a["astride"] == 1:
                F.fp16_conv_dgrad_wf_m(a["desc"], t(a["dy"]), t(a["wf"]), t(a["addend"]),
                                       t(a["amask"]), t(a["dx"]), ws)
            else:
                F.fp16_conv_dgrad_wf_ex(a["desc"], t(a["dy"]), t(a["wf"]), t(a["addend"]),
                                        t(a["amask"]), a["astride"], t(a["dx"]), ws)
        elif k == "dgrad_filter":
            F.fp16_conv_dgrad_filter(a["desc"], t(a["w"]), t(a["wf"]))
        elif k == "dgrad_filters":
            F.fp16_conv_dgrad_filters([d for d, _, _ in a["items"]], [t(w) for _, w, _ in a["items"]],
                                      [t(f) for _, _, f in a["items"]])
        elif k == "conv_wgrad":
            F.fp16_conv_wgrad_ex(a["desc"], t(a["x"]), t(a["dy"]), t(a["dw"]), ws,
                                 workgroups=a["wg"])
        elif k == "conv_bn_fwd":
            nm = op.name
            if a["mask"] is None:
                F.fp16_conv_bn_relu_fwd(a["desc"], a["bn"], t(a["x"]), t(a["w"]),
                                        t(nm + ".gamma"), t(nm + ".beta"), t(a["res"]), t(a["y"]),
                                        t(a["z"]), t(a["stats"]), ws)
            else:
                F.fp16_conv_bn_relu_fwd_m(a["desc"], a["bn"], t(a["x"]), t(a["w"]),
                                          t(nm + ".gamma"), t(nm + ".beta"), t(a["res"]),
                                          t(a["y"]), t(a["z"]), t(a["stats"]), t(a["mask"]), ws)
        elif k == "bn_fwd":
            nm = op.name
            if a["mask"] is None:
                F.fp16_bn_relu(a["desc"], t(a["x"]), t(nm + ".gamma"), t(nm + ".beta"),
                               t(a["res"]), t(a["y"]), t(a["stats"]), ws)
            else:
                F.fp16_bn_relu_m(a["desc"], t(a["x"]), t(nm + ".gamma"), t(nm + ".beta"),
                                 t(a["res"]), t(a["y"]), t(a["stats"]), t(a["mask"]), ws)
        elif k == "bn_bwd":
            nm = op.name
            if a["mask"] is None:
                F.fp16_bn_relu_bwd(a["desc"], t(a["x"]), t(a["y"]), t(a["dy"]), t(nm + ".gamma"),
                                   t(nm + ".beta"), t(a["res"]), t(a["stats"]), t(a["dx"]),
                                   t(a["dgamma"]), t(a["dbeta"]), t(a["dres"]), ws)
            else:
                F.fp16_bn_relu_bwd_m(a["desc"], t(a["x"]), t(a["mask"]), t(a["dy"]),
                                     t(nm + ".gamma"), t(nm + ".beta"), t(a["stats"]), t(a["dx"]),
                                     t(a["dgamma"]), t(a["dbeta"]), t(a["dres"]), ws)
        elif k == "maxpool_fwd":
            F.fp16_maxpool_fwd(a["desc"], t(a["x"]), t(a["y"]), t(a["idx"]))
        elif k == "bn_maxpool_fwd":
            nm = op.name
            F.fp16_bn_relu_maxpool(a["desc"], a["pool"], t(a["x"]), t(nm + ".gamma"),
                                   t(nm + ".beta"), t(a["stats"]), t(a["y"]), t(a["idx"]), ws)
        elif k == "maxpool_bwd":
            F.fp16_maxpool_bwd(a["desc"], t(a["idx"]), t(a["dy"]), t(a["dx"]))
        elif k == "avgpool_fwd":
            F.fp16_avgpool_fwd(a["desc"], t(a["x"]), t(a["y"]))
        elif k == "avgpool_bwd":
            F.fp16_avgpool_bwd(a["desc"], t(a["dy"]), t(a["dx"]))
        elif k == "softmax_ce":
            F.fp16_softmax_ce(a["n"], a["k"], t(a["z"]), t(a["bias"]), t(a["labels"]),
                              t(a["loss"]), t(a["dz"]), t(a["dbias"]))
        elif k == "sgd":
            F.fp16_sgd_step(a["w"], a["g"], a["m"], a["w"].numel(), self.lr, self.momentum,
                            a["wd"])
        else:
            raise ValueError(k)

    @property
    def prep_op(self):
        """The rearrangements of self.prep as one batched call."""
        return Op("dgrad_filters", "prep", {"items": [(o.a["desc"], o.a["w"], o.a["wf"])
                                                      for o in self.prep]})

    def program(self):
        return [self.prep_op] + self.fwd + self.bwd + self.upd

    _OUTPUTS = {"conv_fwd": ("y",), "conv_bn_fwd": ("y", "z", "stats", "mask"),
                "conv_dgrad": ("dx",), "conv_dgrad_add": ("dx",),
                "conv_wgrad": ("dw",), "bn_fwd": ("y", "stats", "mask"),
                "bn_bwd": ("dx", "dgamma", "dbeta", "dres"), "maxpool_fwd": ("y", "idx"),
                "maxpool_bwd": ("dx",), "avgpool_fwd": ("y",), "avgpool_bwd": ("dx",),
                "bn_maxpool_fwd": ("stats", "y", "idx"),
                "softmax_ce": ("loss", "dz", "dbias"), "dgrad_filter": ("wf",)}

    def _schedule(self):
        """For each weight gradient of the backward, the index (in bwd) of the
        call that writes its input gradient, or -1 when that happens before the
        backward starts; and for each fused downsampling shortcut of the
        forward, the index of its block's first call (where it can start)."""
        self._fwd_branch = {}
        for i, op in enumerate(self.fwd):
            if op.kind == "conv_bn_fwd" and op.a["conv"].endswith(".ds"):
                first = min(j for j, o in enumerate(self.fwd) if o.a.get("x") == op.a["x"])
                self._fwd_branch[first] = i
        self._fwd_skip = set(self._fwd_branch.values())
        writer = {}
        self._dep = {}
        self._mark = set()
        for i, op in enumerate(self.bwd):
            if op.kind == "conv_wgrad":
                dep = writer.get(op.a["dy"], -1)
                self._dep[i] = dep
                if dep >= 0:
                    self._mark.add(dep)
            else:
                for k in self._OUTPUTS[op.kind]:
                    if op.a.get(k) is not None:
                        writer[op.a[k]] = i

    def forward(self):
        # the data-gradient filters of this step's weights, on the side stream
        # while the forward runs (the backward waits for them)
        # (all of them in one call: launched one filter each, they ran one
        # after another ahead of the forward, 0.54 ms of the step)
        if self.side is None:
            self.run(self.prep_op)
        else:
            main = torch.cuda.current_stream()
            start = torch.cuda.Event()
            start.record(main)
            self.side.wait_event(start)
            with torch.cuda.stream(self.side):
                self.run(self.prep_op, ws=self.ws_side)
            self._wf_ready = torch.cuda.Event()
            self._wf_ready.record(self.side)
        if self.side is None:
            for op in self.fwd:
                self.run(op)
            return
        # a downsampling block's shortcut (its conv + BN, one call) runs on the
        # side stream from the block input on, beside the block's first two
        # convolutions; the block-last BN, which adds it, waits for it
        done = {}
        for i, op in enumerate(self.fwd):
            if i in self._fwd_branch:
                ev = torch.cuda.Event()
                ev.record(main)
                self.side.wait_event(ev)
                br = self.fwd[self._fwd_branch[i]]
                with torch.cuda.stream(self.side):
                    self.run(br, ws=self.ws_side)
                done[br.a["z"]] = torch.cuda.Event()
                done[br.a["z"]].record(self.side)
            if i in self._fwd_skip:
                continue
            if op.a.get("res") in done:
                main.wait_event(done[op.a["res"]])
            self.run(op)

    def backward(self):
        if self.side is None:
            for op in self.bwd:
                self.run(op)
            return
        main, side = torch.cuda.current_stream(), self.side
        main.wait_event(self._wf_ready)  # the rearranged data-gradient filters
        start = torch.cuda.Event()
        start.record(main)
        events = {}
        for i, op in enumerate(self.bwd):
            if op.kind == "conv_wgrad":
                dep = self._dep[i]
                side.wait_event(events[dep] if dep >= 0 else start)
                with torch.cuda.stream(side):
                    self.run(op, ws=self.ws_side)
            else:
                self.run(op)
                if i in self._mark:
                    ev = torch.cuda.Event()
                    ev.record(main)
                    events[i] = ev
        main.wait_stream(side)  # the update reads every weight gradient

    def update(self):
        for op in self.upd:
            self.run(op)

    def step(self):
        self.forward()
        self.backward()
        self.update()

    def calls(self):
        """(name, thunk) for every ABI call of one step, in order."""
        return [(f"{op.name}:{op.kind}", (lambda o=op: self.run(o))) for op in self.program()]

    # ---- accounting -----------------------------------------------------------------

    def conv_flops(self) -> int:
        """Algorithmic FLOPs of one forward pass over every convolution (the
        classifier included); a training step does three such passes, less the
        stem's data gradient, which is not computed."""
        tot = 0
        for c in self.convs:
            d = c["desc"]
            p, q = F.fp16_conv_out_dims(d)
            tot += 2 * d.n * p * q * d.k * d.c * d.r * d.s
        return tot

    def step_flops(self) -> int:
        stem = next(c for c in self.convs if c["name"] == "stem")["desc"]
        p, q = F.fp16_conv_out_dims(stem)
        return 3 * self.conv_flops() - 2 * stem.n * p * q * stem.k * stem.c * stem.r * stem.s

    def state(self):
        return [t.clone() for t in (self.w_arena, self.mw_arena, self.bn_arena, self.mbn_arena)]

    def load_state(self, st):
        for t, v in zip((self.w_arena, self.mw_arena, self.bn_arena, self.mbn_arena), st):
            t.copy_(v)
