"""Helpers for the GPU parity tests: run a pass through the C ABI on seeded
inputs and compare with the oracle on the same binary16 bytes."""

from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
import paper_1911_07384_amd as F
from paper_1911_07384_amd import synth


def require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU test selected but no GPU is visible")


def dev(a) -> torch.Tensor:
    """Host float16/uint16 array -> contiguous float16 device tensor (same bits)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.float16)
    return torch.from_numpy(a).to("cuda")


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def note(msg: str) -> None:
    """Name the case before a GPU step (flushed, so a fault still shows it)."""
    print(msg, file=sys.stderr, flush=True)


def ulp_dist(a16: np.ndarray, b16: np.ndarray) -> np.ndarray:
    """Distance in units in the last place between two binary16 arrays
    (ordered-integer distance; +0 and -0 are the same value)."""
    def ordered(x):
        b = np.ascontiguousarray(x).view(np.uint16).astype(np.int32)
        return np.where(b & 0x8000, -(b & 0x7FFF), b)
    return np.abs(ordered(a16) - ordered(b16))


class ConvCase:
    """One convolution problem with seeded inputs (x ~ N(0,1), He-normal W,
    dy ~ N(0, dy_std^2)) and the three passes on the GPU."""

    def __init__(self, n, c, h, w, k, r, s, stride=1, pad=0, layout="NHWC", seed=0,
                 dy_std=1e-2, x=None, wt=None, dy=None, accum=0):
        self.shp = oracle.conv_shape(n, c, h, w, k, r, s, stride, pad, layout)
        self.desc = F.conv_desc(n, c, h, w, k, r, s, stride, pad, layout, accum=accum)
        self.P, self.Q = F.fp16_conv_out_dims(self.desc)
        assert (self.P, self.Q) == oracle.conv_out_dims(self.shp)
        if layout == "NHWC":
            xs, ws, ys = (n, h, w, c), (k, r, s, c), (n, self.P, self.Q, k)
        else:
            xs, ws, ys = (n, c, h, w), (k, c, r, s), (n, k, self.P, self.Q)
        self.xs, self.ws, self.ys = xs, ws, ys
        self.x = synth.normal_f16(xs, 1.0, seed, 1) if x is None else x
        self.w = synth.normal_f16(ws, synth.he_std(c * r * s), seed, 2) if wt is None else wt
        self.dy = synth.normal_f16(ys, dy_std, seed, 3) if dy is None else dy
        assert self.x.shape == xs and self.w.shape == ws and self.dy.shape == ys
        self.label = f"conv n={n} c={c} hw={h}x{w} k={k} rs={r}x{s} st={stride} pad={pad} {layout}"

    def run(self, which, workgroups=None):
        """One pass on the GPU; workgroups (weight gradient only) goes through
        fp16_conv_wgrad_ex."""
        x, w, dy = dev(self.x), dev(self.w), dev(self.dy)
        pass_ = {"fwd": F.PASS_FWD, "dgrad": F.PASS_DGRAD, "wgrad": F.PASS_WGRAD}[which]
        ws = F.workspace(F.fp16_conv_workspace_bytes(self.desc, pass_))
        note(f"[gpu] {which} {self.label}")
        if which == "fwd":
            out = torch.empty(self.ys, dtype=torch.float16, device="cuda")
            F.fp16_conv_fwd(self.desc, x, w, out, ws)
        elif which == "dgrad":
            out = torch.empty(self.xs, dtype=torch.float16, device="cuda")
            F.fp16_conv_dgrad(self.desc, dy, w, out, ws)
        else:
            out = torch.empty(self.ws, dtype=torch.float16, device="cuda")
            if workgroups is None:
                F.fp16_conv_wgrad(self.desc, x, dy, out, ws)
            else:
                F.fp16_conv_wgrad_ex(self.desc, x, dy, out, ws, workgroups=workgroups)
        torch.cuda.synchronize()
        return host(out)

    def oracle(self, which):
        if which == "fwd":
            return oracle.conv_fwd(self.shp, self.x, self.w)
        if which == "dgrad":
            return oracle.conv_dgrad(self.shp, self.dy, self.w)
        return oracle.conv_wgrad(self.shp, self.x, self.dy)

    def oracle_at(self, which, idx):
        if which == "fwd":
            return oracle.conv_fwd_at(self.shp, self.x, self.w, idx)
        if which == "dgrad":
            return oracle.conv_dgrad_at(self.shp, self.dy, self.w, idx)
        return oracle.conv_wgrad_at(self.shp, self.x, self.dy, idx)


def check_close(got16: np.ndarray, ref64: np.ndarray, rel=1e-2, what=""):
    """Parity bar for the convolutions: max |gpu - ref| <= rel * RMS(ref)."""
    g = got16.astype(np.float64)
    assert g.shape == ref64.shape, (g.shape, ref64.shape)
    assert np.all(np.isfinite(g)), what
    rms = float(np.sqrt(np.mean(ref64 ** 2)))
    err = float(np.max(np.abs(g - ref64))) if g.size else 0.0
    assert err <= rel * rms or (rms == 0.0 and err == 0.0), f"{what}: max err {err:.3e} > {rel} * RMS {rms:.3e}"
    return err, rms
