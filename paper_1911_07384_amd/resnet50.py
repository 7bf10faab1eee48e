"""ResNet-50 convolution geometry (torchvision v1.5: stride on the 3x3 conv of
each downsampling bottleneck) -- the network of Section 5.1 of
arXiv:1911.07384 -- and a per-layer timing sweep of the three convolution
passes through the C ABI.

The 53 convolutions reduce to 23 distinct shapes; each is listed once with
its multiplicity in the network.
"""

from __future__ import annotations

from dataclasses import dataclass

import torch

import paper_1911_07384_amd as F


@dataclass(frozen=True)
class ConvLayer:
    name: str
    c: int
    k: int
    r: int
    stride: int
    hw: int      # input spatial size
    mult: int    # occurrences in the network

    @property
    def pad(self) -> int:
        return self.r // 2

    @property
    def out_hw(self) -> int:
        return (self.hw + 2 * self.pad - self.r) // self.stride + 1

    def flops(self, n: int) -> int:
        """Algorithmic FLOPs of one pass (2 per multiply-add)."""
        return 2 * n * self.out_hw ** 2 * self.k * self.c * self.r * self.r


# name, C, K, R, stride, input H=W, multiplicity
LAYERS = [
    ConvLayer("conv1 (stem)", 3, 64, 7, 2, 224, 1),
    ConvLayer("l1.0.c1", 64, 64, 1, 1, 56, 1),
    ConvLayer("l1.*.c2", 64, 64, 3, 1, 56, 3),
    ConvLayer("l1.*.c3 / l1.0.ds", 64, 256, 1, 1, 56, 4),
    ConvLayer("l1.{1,2}.c1", 256, 64, 1, 1, 56, 2),
    ConvLayer("l2.0.c1", 256, 128, 1, 1, 56, 1),
    ConvLayer("l2.0.c2", 128, 128, 3, 2, 56, 1),
    ConvLayer("l2.*.c3", 128, 512, 1, 1, 28, 4),
    ConvLayer("l2.0.ds", 256, 512, 1, 2, 56, 1),
    ConvLayer("l2.{1-3}.c1", 512, 128, 1, 1, 28, 3),
    ConvLayer("l2.{1-3}.c2", 128, 128, 3, 1, 28, 3),
    ConvLayer("l3.0.c1", 512, 256, 1, 1, 28, 1),
    ConvLayer("l3.0.c2", 256, 256, 3, 2, 28, 1),
    ConvLayer("l3.*.c3", 256, 1024, 1, 1, 14, 6),
    ConvLayer("l3.0.ds", 512, 1024, 1, 2, 28, 1),
    ConvLayer("l3.{1-5}.c1", 1024, 256, 1, 1, 14, 5),
    ConvLayer("l3.{1-5}.c2", 256, 256, 3, 1, 14, 5),
    ConvLayer("l4.0.c1", 1024, 512, 1, 1, 14, 1),
    ConvLayer("l4.0.c2", 512, 512, 3, 2, 14, 1),
    ConvLayer("l4.*.c3", 512, 2048, 1, 1, 7, 3),
    ConvLayer("l4.0.ds", 1024, 2048, 1, 2, 14, 1),
    ConvLayer("l4.{1,2}.c1", 2048, 512, 1, 1, 7, 2),
    ConvLayer("l4.{1,2}.c2", 512, 512, 3, 1, 7, 2),
]

assert sum(l.mult for l in LAYERS) == 53


def sweep(n: int = 128, layers=None, reps: int = 10, seed: int = 0, passes=("fwd", "dgrad", "wgrad"),
          layout: str = "NHWC"):
    """Time each convolution pass of each layer shape at batch n.

    Inputs are seeded device tensors (x ~ N(0,1), He-normal W, dy ~ N(0, 1e-3^2)),
    NHWC/KRSC or NCHW/KCRS.  Each pass is timed over `reps` back-to-back calls
    between two HIP events on the launch stream, after one untimed call.
    Returns a list of dicts."""
    layers = LAYERS if layers is None else layers
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    out = []
    for L in layers:
        p = L.out_hw
        d = F.conv_desc(n, L.c, L.hw, L.hw, L.k, L.r, L.r, L.stride, L.pad, layout)
        if layout == "NHWC":
            xs, ws_, ys = (n, L.hw, L.hw, L.c), (L.k, L.r, L.r, L.c), (n, p, p, L.k)
        else:
            xs, ws_, ys = (n, L.c, L.hw, L.hw), (L.k, L.c, L.r, L.r), (n, L.k, p, p)
        x = torch.randn(xs, generator=gen, device="cuda").half()
        w = (torch.randn(ws_, generator=gen, device="cuda") * (2.0 / (L.c * L.r * L.r)) ** 0.5).half()
        dy = (torch.randn(ys, generator=gen, device="cuda") * 1e-3).half()
        y = torch.empty(ys, dtype=torch.float16, device="cuda")
        dx = torch.empty_like(x)
        dw = torch.empty_like(w)
        ws = F.workspace(max(F.fp16_conv_workspace_bytes(d, q) for q in (0, 1, 2)))
        fns = {"fwd": lambda: F.fp16_conv_fwd(d, x, w, y, ws),
               "dgrad": lambda: F.fp16_conv_dgrad(d, dy, w, dx, ws),
               "wgrad": lambda: F.fp16_conv_wgrad(d, x, dy, dw, ws)}
        row = {"layer": L.name, "c": L.c, "k": L.k, "r": L.r, "stride": L.stride, "hw": L.hw,
               "mult": L.mult, "gflop": L.flops(n) / 1e9}
        for name in passes:
            fn = fns[name]
            fn()
            torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(2_000_000)  # queue the calls before they start
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            torch.cuda.synchronize()
            ms = a.elapsed_time(b) / reps
            row[name + "_us"] = ms * 1e3
            row[name + "_tflops"] = L.flops(n) / (ms * 1e-3) / 1e12
        out.append(row)
        del x, w, dy, y, dx, dw, ws
    return out


def summarize(rows, peak_tflops: float, passes=("fwd", "dgrad", "wgrad")):
    """Network-weighted totals: time and FLOPs of every layer x multiplicity."""
    def agg(sel):
        t = sum(r[p + "_us"] * r["mult"] for r in rows if sel(r) for p in passes) * 1e-6
        f = sum(r["gflop"] * 1e9 * r["mult"] * len(passes) for r in rows if sel(r))
        return {"tflop": f / 1e12, "ms": t * 1e3, "tflops": f / t / 1e12 if t else 0.0,
                "pct_mfma_peak": 100 * f / t / 1e12 / peak_tflops if t else 0.0}
    return {"all_53": agg(lambda r: True), "3x3_16": agg(lambda r: r["r"] == 3)}
