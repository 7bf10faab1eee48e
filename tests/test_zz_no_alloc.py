"""The weight gradient without a workspace argument (fp16_conv_wgrad_noalloc,
for callers that cannot allocate): called through the C ABI, its output is
bit-identical to fp16_conv_wgrad's on the same inputs -- two calls in a row
on the library's device-resident scratch, the second with a smaller problem
(so stale partial sums of the first would show) -- and a problem whose
scratch need exceeds the stated maximum is refused before anything runs."""

import ctypes

import numpy as np
import pytest
import torch

import paper_1911_07384_amd as F
from gpu_util import dev, host, note, require_gpu
from paper_1911_07384_amd import synth

pytestmark = pytest.mark.gpu

# (n, c, hw, k, r, stride, pad): the conv2_x 3x3 layer at batch 16, then a
# smaller stride-2 1x1 problem with fewer splits and a narrower filter
CASES = [(16, 64, 56, 64, 3, 1, 1), (2, 256, 14, 128, 1, 2, 0)]


def _inputs(n, c, hw, k, r, stride, pad, seed):
    d = F.conv_desc(n, c, hw, hw, k, r, r, stride, pad)
    p, q = F.fp16_conv_out_dims(d)
    x = synth.normal_f16((n, hw, hw, c), 1.0, seed, 1)
    dy = synth.normal_f16((n, p, q, k), 1e-2, seed, 3)
    return d, x, dy


def test_noalloc_matches_workspace_call_twice():
    require_gpu()
    lib = F.lib()
    stream = torch.cuda.current_stream().cuda_stream
    for i, (n, c, hw, k, r, stride, pad) in enumerate(CASES):
        d, x, dy = _inputs(n, c, hw, k, r, stride, pad, 80 + i)
        assert F.fp16_conv_workspace_bytes(d, F.PASS_WGRAD) <= lib.fp16_noalloc_scratch_bytes()
        X, DY = dev(x), dev(dy)
        ref = torch.empty((k, r, r, c), dtype=torch.float16, device="cuda")
        got = torch.full((k, r, r, c), float("nan"), dtype=torch.float16, device="cuda")
        ws = F.workspace(F.fp16_conv_workspace_bytes(d, F.PASS_WGRAD))
        note(f"[gpu] wgrad noalloc call {i}: n={n} c={c} hw={hw} k={k} r={r} stride={stride}")
        F.fp16_conv_wgrad(d, X, DY, ref, ws)
        st = lib.fp16_conv_wgrad_noalloc(ctypes.byref(d), X.data_ptr(), DY.data_ptr(),
                                         got.data_ptr(), stream)
        assert st == 0, F.fp16_status_string(st)
        torch.cuda.synchronize()
        assert np.array_equal(host(got).view(np.uint16), host(ref).view(np.uint16)), i


def test_noalloc_refuses_oversized_problem():
    require_gpu()
    lib = F.lib()
    # the ResNet stem's weight gradient at batch 128 needs 81 MiB of scratch
    d = F.conv_desc(128, 3, 224, 224, 64, 7, 7, 2, 3)
    assert F.fp16_conv_workspace_bytes(d, F.PASS_WGRAD) > lib.fp16_noalloc_scratch_bytes()
    t = torch.zeros(16, dtype=torch.float16, device="cuda")
    st = lib.fp16_conv_wgrad_noalloc(ctypes.byref(d), t.data_ptr(), t.data_ptr(), t.data_ptr(),
                                     None)
    assert st == 6  # FP16_ERR_WORKSPACE
