"""paper_1911_07384_amd: the all-FP16 training hot path of arXiv:1911.07384
("Distributed low-precision Training Without Mixed Precision") on MI355X.

This module is a thin ctypes binding over ``libfp16train.so``, whose C ABI is
declared in ``include/fp16train.h``.  Functions carry the same names as the
C entry points and only marshal arguments: torch tensors (float16, CUDA/HIP
device, contiguous) are passed as raw device pointers, and work is enqueued
on the current torch stream unless another stream is given.  Every step of
the computation runs in the HIP kernels; there is no fallback path.  A
nonzero status raises ``Fp16Error``.
"""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfp16train.so")

FP16_NHWC = 0
FP16_NCHW = 1
PASS_FWD, PASS_DGRAD, PASS_WGRAD = 0, 1, 2
_LAYOUTS = {"NHWC": FP16_NHWC, "NCHW": FP16_NCHW, FP16_NHWC: FP16_NHWC, FP16_NCHW: FP16_NCHW}

STATUS = {0: "FP16_OK", 1: "FP16_ERR_NULL", 2: "FP16_ERR_SHAPE", 3: "FP16_ERR_LAYOUT",
          4: "FP16_ERR_MISALIGNED", 5: "FP16_ERR_ALIASING", 6: "FP16_ERR_WORKSPACE",
          7: "FP16_ERR_UNSUPPORTED", 8: "FP16_ERR_HIP"}

EXPORTS = ["fp16_conv_out_dims", "fp16_conv_workspace_bytes", "fp16_conv_fwd", "fp16_conv_dgrad",
           "fp16_conv_dgrad_add", "fp16_conv_wgrad", "fp16_bn_workspace_bytes", "fp16_bn_relu", "fp16_bn_relu_bwd",
           "fp16_sgd_step", "fp16_pool_out_dims", "fp16_maxpool_fwd", "fp16_maxpool_bwd",
           "fp16_avgpool_fwd", "fp16_avgpool_bwd", "fp16_softmax_ce", "fp16_status_string",
           "fp16_version", "fp16_conv_bn_workspace_bytes", "fp16_conv_bn_relu_fwd",
           "fp16_sgd_step_f16", "fp16_conv_dgrad_filter_bytes", "fp16_conv_dgrad_filter",
           "fp16_conv_dgrad_filters",
           "fp16_conv_dgrad_wf", "fp16_noalloc_scratch_bytes", "fp16_conv_wgrad_noalloc",
           "fp16_bn_mask_bytes", "fp16_bn_relu_m", "fp16_bn_relu_bwd_m", "fp16_conv_bn_relu_fwd_m",
           "fp16_conv_dgrad_wf_m", "fp16_bn_relu_maxpool", "fp16_conv_wgrad_ex",
           "fp16_conv_dgrad_wf_ex"]


class Fp16Error(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn}: {STATUS.get(status, status)} ({_status_string(status)})")


class ConvDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n", "c", "h", "w", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w",
                 "layout", "accum")]


class BnDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("c", ctypes.c_int32), ("h", ctypes.c_int32),
                ("w", ctypes.c_int32), ("layout", ctypes.c_int32), ("eps", ctypes.c_float),
                ("post_scale", ctypes.c_float), ("relu", ctypes.c_int32),
                ("use_stats", ctypes.c_int32), ("swap", ctypes.c_int32)]


class PoolDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n", "c", "h", "w", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w", "layout")]


_lib = None
_P = ctypes.c_void_p
_SZ = ctypes.c_size_t
_F = ctypes.c_float
_I32 = ctypes.c_int32
_SIGS = {
    "fp16_conv_out_dims": (ctypes.c_int, [_P, _P, _P]),
    "fp16_conv_workspace_bytes": (_SZ, [_P, _I32]),
    "fp16_conv_fwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _SZ, _P]),
    "fp16_conv_dgrad": (ctypes.c_int, [_P, _P, _P, _P, _P, _SZ, _P]),
    "fp16_conv_dgrad_add": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _SZ, _P]),
    "fp16_conv_wgrad": (ctypes.c_int, [_P, _P, _P, _P, _P, _SZ, _P]),
    "fp16_conv_dgrad_filter_bytes": (_SZ, [_P]),
    "fp16_noalloc_scratch_bytes": (_SZ, []),
    "fp16_conv_wgrad_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _P]),
    "fp16_conv_dgrad_filter": (ctypes.c_int, [_P, _P, _P, _P]),
    "fp16_conv_dgrad_filters": (ctypes.c_int, [ctypes.c_int32, _P, _P, _P, _P]),
    "fp16_conv_dgrad_wf": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _SZ, _P]),
    "fp16_conv_dgrad_wf_m": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "fp16_bn_relu_maxpool": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "fp16_conv_wgrad_ex": (ctypes.c_int, [_P, _P, _P, _P, _P, _SZ, ctypes.c_int32, _P]),
    "fp16_conv_dgrad_wf_ex": (ctypes.c_int, [_P, _P, _P, _P, _P, ctypes.c_int32, _P, _P, _SZ, _P]),
    "fp16_bn_workspace_bytes": (_SZ, [_P]),
    "fp16_bn_mask_bytes": (_SZ, [_P]),
    "fp16_bn_relu_m": (ctypes.c_int, [_P] * 9 + [_SZ, _P]),
    "fp16_bn_relu_bwd_m": (ctypes.c_int, [_P] * 12 + [_SZ, _P]),
    "fp16_conv_bn_relu_fwd_m": (ctypes.c_int, [_P] * 12 + [_SZ, _P]),
    "fp16_bn_relu": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "fp16_bn_relu_bwd": (ctypes.c_int, [_P] * 13 + [_SZ, _P]),
    "fp16_sgd_step": (ctypes.c_int, [_P, _P, _P, _SZ, _F, _F, _F, _P]),
    "fp16_sgd_step_f16": (ctypes.c_int, [_P, _P, _P, _SZ, _F, _F, _F, _P]),
    "fp16_pool_out_dims": (ctypes.c_int, [_P, _P, _P]),
    "fp16_maxpool_fwd": (ctypes.c_int, [_P, _P, _P, _P, _P]),
    "fp16_maxpool_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P]),
    "fp16_avgpool_fwd": (ctypes.c_int, [_P, _P, _P, _P]),
    "fp16_avgpool_bwd": (ctypes.c_int, [_P, _P, _P, _P]),
    "fp16_softmax_ce": (ctypes.c_int, [_I32, _I32, _P, _P, _P, _P, _P, _P, _P]),
    "fp16_conv_bn_workspace_bytes": (_SZ, [_P, _P]),
    "fp16_conv_bn_relu_fwd": (ctypes.c_int, [_P] * 11 + [_SZ, _P]),
    "fp16_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "fp16_version": (ctypes.c_char_p, []),
}


def lib() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -c 'import "
                               f"__graft_entry__ as g; g.build()'` (no fallback path exists)")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def _status_string(status: int) -> str:
    try:
        return lib().fp16_status_string(int(status)).decode()
    except Exception:  # pragma: no cover - only when the library cannot load
        return "?"


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise Fp16Error(fn, status)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    import torch
    if t.dtype not in (torch.float16, torch.float32, torch.uint8, torch.int32):
        raise TypeError(f"expected float16/float32/uint8/int32 tensor, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def conv_desc(n, c, h, w, k, r, s, stride=1, pad=0, layout="NHWC", accum=0) -> ConvDesc:
    """accum = 1 selects binary16 accumulation (see fp16_conv_desc.accum)."""
    sh, sw = (stride, stride) if isinstance(stride, int) else stride
    ph, pw = (pad, pad) if isinstance(pad, int) else pad
    return ConvDesc(n, c, h, w, k, r, s, sh, sw, ph, pw, _LAYOUTS[layout], int(accum))


def bn_desc(n, c, h, w, layout="NHWC", eps=1e-5, post_scale=1.0, relu=True, use_stats=False,
            swap=False) -> BnDesc:
    return BnDesc(n, c, h, w, _LAYOUTS[layout], eps, post_scale, int(bool(relu)),
                  int(bool(use_stats)), int(bool(swap)))


# ---- C entry points, same names --------------------------------------------

def fp16_version() -> str:
    return lib().fp16_version().decode()


def fp16_status_string(status: int) -> str:
    return lib().fp16_status_string(int(status)).decode()


def fp16_conv_out_dims(desc: ConvDesc):
    p, q = ctypes.c_int32(), ctypes.c_int32()
    _check("fp16_conv_out_dims", lib().fp16_conv_out_dims(ctypes.byref(desc), ctypes.byref(p),
                                                          ctypes.byref(q)))
    return p.value, q.value


def fp16_conv_workspace_bytes(desc: ConvDesc, pass_: int) -> int:
    return int(lib().fp16_conv_workspace_bytes(ctypes.byref(desc), int(pass_)))


def fp16_conv_fwd(desc, x, w, y, ws=None, ws_bytes=None, stream=None) -> None:
    _check("fp16_conv_fwd", lib().fp16_conv_fwd(ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(y),
                                                _ptr(ws), _wsb(ws, ws_bytes), _stream(stream)))


def fp16_conv_dgrad(desc, dy, w, dx, ws=None, ws_bytes=None, stream=None) -> None:
    _check("fp16_conv_dgrad", lib().fp16_conv_dgrad(ctypes.byref(desc), _ptr(dy), _ptr(w), _ptr(dx),
                                                    _ptr(ws), _wsb(ws, ws_bytes), _stream(stream)))


def fp16_conv_dgrad_add(desc, dy, w, addend, dx, ws=None, ws_bytes=None, stream=None) -> None:
    _check("fp16_conv_dgrad_add", lib().fp16_conv_dgrad_add(
        ctypes.byref(desc), _ptr(dy), _ptr(w), _ptr(addend), _ptr(dx), _ptr(ws), _wsb(ws, ws_bytes),
        _stream(stream)))


def fp16_conv_dgrad_filter_bytes(desc: ConvDesc) -> int:
    return int(lib().fp16_conv_dgrad_filter_bytes(ctypes.byref(desc)))


def fp16_conv_dgrad_filter(desc, w, wf, stream=None) -> None:
    _check("fp16_conv_dgrad_filter", lib().fp16_conv_dgrad_filter(ctypes.byref(desc), _ptr(w),
                                                                  _ptr(wf), _stream(stream)))


def fp16_conv_dgrad_filters(descs, ws, wfs, stream=None) -> None:
    """fp16_conv_dgrad_filter for every (desc, w, wf) of the three lists."""
    n = len(descs)
    if not (len(ws) == len(wfs) == n):
        raise ValueError("descs, ws and wfs differ in length")
    d = (ConvDesc * max(n, 1))(*descs)
    w = (ctypes.c_void_p * max(n, 1))(*[_ptr(t) for t in ws])
    f = (ctypes.c_void_p * max(n, 1))(*[_ptr(t) for t in wfs])
    _check("fp16_conv_dgrad_filters", lib().fp16_conv_dgrad_filters(n, d, w, f, _stream(stream)))


def fp16_conv_dgrad_wf(desc, dy, wf, addend, dx, ws=None, ws_bytes=None, stream=None) -> None:
    _check("fp16_conv_dgrad_wf", lib().fp16_conv_dgrad_wf(
        ctypes.byref(desc), _ptr(dy), _ptr(wf), _ptr(addend), _ptr(dx), _ptr(ws),
        _wsb(ws, ws_bytes), _stream(stream)))


def fp16_conv_dgrad_wf_m(desc, dy, wf, addend, mask, dx, ws=None, ws_bytes=None,
                         stream=None) -> None:
    _check("fp16_conv_dgrad_wf_m", lib().fp16_conv_dgrad_wf_m(
        ctypes.byref(desc), _ptr(dy), _ptr(wf), _ptr(addend), _ptr(mask), _ptr(dx), _ptr(ws),
        _wsb(ws, ws_bytes), _stream(stream)))


def fp16_conv_dgrad_wf_ex(desc, dy, wf, addend, mask, addend_stride, dx, ws=None, ws_bytes=None,
                          stream=None) -> None:
    _check("fp16_conv_dgrad_wf_ex", lib().fp16_conv_dgrad_wf_ex(
        ctypes.byref(desc), _ptr(dy), _ptr(wf), _ptr(addend), _ptr(mask), int(addend_stride),
        _ptr(dx), _ptr(ws), _wsb(ws, ws_bytes), _stream(stream)))


def fp16_conv_wgrad(desc, x, dy, dw, ws=None, ws_bytes=None, stream=None) -> None:
    _check("fp16_conv_wgrad", lib().fp16_conv_wgrad(ctypes.byref(desc), _ptr(x), _ptr(dy), _ptr(dw),
                                                    _ptr(ws), _wsb(ws, ws_bytes), _stream(stream)))


def fp16_conv_wgrad_ex(desc, x, dy, dw, ws=None, ws_bytes=None, workgroups=0,
                       stream=None) -> None:
    _check("fp16_conv_wgrad_ex", lib().fp16_conv_wgrad_ex(
        ctypes.byref(desc), _ptr(x), _ptr(dy), _ptr(dw), _ptr(ws), _wsb(ws, ws_bytes),
        int(workgroups), _stream(stream)))


def fp16_noalloc_scratch_bytes() -> int:
    return int(lib().fp16_noalloc_scratch_bytes())


def fp16_conv_wgrad_noalloc(desc, x, dy, dw, stream=None) -> None:
    _check("fp16_conv_wgrad_noalloc", lib().fp16_conv_wgrad_noalloc(
        ctypes.byref(desc), _ptr(x), _ptr(dy), _ptr(dw), _stream(stream)))


def fp16_bn_workspace_bytes(desc: BnDesc) -> int:
    return int(lib().fp16_bn_workspace_bytes(ctypes.byref(desc)))


def fp16_bn_relu(desc, x, gamma, beta, residual, y, stats, ws=None, ws_bytes=None,
                 stream=None) -> None:
    _check("fp16_bn_relu", lib().fp16_bn_relu(ctypes.byref(desc), _ptr(x), _ptr(gamma), _ptr(beta),
                                              _ptr(residual), _ptr(y), _ptr(stats), _ptr(ws),
                                              _wsb(ws, ws_bytes), _stream(stream)))


def fp16_bn_relu_bwd(desc, x, y, dy, gamma, beta, residual, stats, dx, dgamma, dbeta, dresidual,
                     ws=None, ws_bytes=None, stream=None) -> None:
    _check("fp16_bn_relu_bwd", lib().fp16_bn_relu_bwd(
        ctypes.byref(desc), _ptr(x), _ptr(y), _ptr(dy), _ptr(gamma), _ptr(beta), _ptr(residual),
        _ptr(stats), _ptr(dx), _ptr(dgamma), _ptr(dbeta), _ptr(dresidual), _ptr(ws),
        _wsb(ws, ws_bytes), _stream(stream)))


def fp16_bn_mask_bytes(desc: BnDesc) -> int:
    return int(lib().fp16_bn_mask_bytes(ctypes.byref(desc)))


def fp16_bn_relu_m(desc, x, gamma, beta, residual, y, stats, mask, ws=None, ws_bytes=None,
                   stream=None) -> None:
    _check("fp16_bn_relu_m", lib().fp16_bn_relu_m(
        ctypes.byref(desc), _ptr(x), _ptr(gamma), _ptr(beta), _ptr(residual), _ptr(y), _ptr(stats),
        _ptr(mask), _ptr(ws), _wsb(ws, ws_bytes), _stream(stream)))


def fp16_bn_relu_bwd_m(desc, x, mask, dy, gamma, beta, stats, dx, dgamma, dbeta, dresidual,
                       ws=None, ws_bytes=None, stream=None) -> None:
    _check("fp16_bn_relu_bwd_m", lib().fp16_bn_relu_bwd_m(
        ctypes.byref(desc), _ptr(x), _ptr(mask), _ptr(dy), _ptr(gamma), _ptr(beta), _ptr(stats),
        _ptr(dx), _ptr(dgamma), _ptr(dbeta), _ptr(dresidual), _ptr(ws), _wsb(ws, ws_bytes),
        _stream(stream)))


def fp16_sgd_step(w, g, m, n=None, lr=0.1, momentum=0.9, weight_decay=1e-4, stream=None) -> None:
    if n is None:
        n = w.numel()
    _check("fp16_sgd_step", lib().fp16_sgd_step(_ptr(w), _ptr(g), _ptr(m), int(n), float(lr),
                                                float(momentum), float(weight_decay),
                                                _stream(stream)))


def fp16_sgd_step_f16(w, g, m, n=None, lr=0.1, momentum=0.9, weight_decay=1e-4,
                      stream=None) -> None:
    if n is None:
        n = w.numel()
    _check("fp16_sgd_step_f16", lib().fp16_sgd_step_f16(_ptr(w), _ptr(g), _ptr(m), int(n),
                                                        float(lr), float(momentum),
                                                        float(weight_decay), _stream(stream)))


def pool_desc(n, c, h, w, r, s, stride=1, pad=0, layout="NHWC") -> PoolDesc:
    sh, sw = (stride, stride) if isinstance(stride, int) else stride
    ph, pw = (pad, pad) if isinstance(pad, int) else pad
    return PoolDesc(n, c, h, w, r, s, sh, sw, ph, pw, _LAYOUTS[layout])


def fp16_pool_out_dims(desc: PoolDesc):
    p, q = ctypes.c_int32(), ctypes.c_int32()
    _check("fp16_pool_out_dims", lib().fp16_pool_out_dims(ctypes.byref(desc), ctypes.byref(p),
                                                          ctypes.byref(q)))
    return p.value, q.value


def fp16_maxpool_fwd(desc, x, y, idx, stream=None) -> None:
    _check("fp16_maxpool_fwd", lib().fp16_maxpool_fwd(ctypes.byref(desc), _ptr(x), _ptr(y),
                                                      _ptr(idx), _stream(stream)))


def fp16_bn_relu_maxpool(bn, pool, x, gamma, beta, stats, y, idx, ws=None, ws_bytes=None,
                         stream=None) -> None:
    _check("fp16_bn_relu_maxpool", lib().fp16_bn_relu_maxpool(
        ctypes.byref(bn), ctypes.byref(pool), _ptr(x), _ptr(gamma), _ptr(beta), _ptr(stats),
        _ptr(y), _ptr(idx), _ptr(ws), _wsb(ws, ws_bytes), _stream(stream)))


def fp16_maxpool_bwd(desc, idx, dy, dx, stream=None) -> None:
    _check("fp16_maxpool_bwd", lib().fp16_maxpool_bwd(ctypes.byref(desc), _ptr(idx), _ptr(dy),
                                                      _ptr(dx), _stream(stream)))


def fp16_avgpool_fwd(desc, x, y, stream=None) -> None:
    _check("fp16_avgpool_fwd", lib().fp16_avgpool_fwd(ctypes.byref(desc), _ptr(x), _ptr(y),
                                                      _stream(stream)))


def fp16_avgpool_bwd(desc, dy, dx, stream=None) -> None:
    _check("fp16_avgpool_bwd", lib().fp16_avgpool_bwd(ctypes.byref(desc), _ptr(dy), _ptr(dx),
                                                      _stream(stream)))


def fp16_softmax_ce(n, k, z, bias, labels, loss, dz, dbias, stream=None) -> None:
    _check("fp16_softmax_ce", lib().fp16_softmax_ce(int(n), int(k), _ptr(z), _ptr(bias),
                                                    _ptr(labels), _ptr(loss), _ptr(dz),
                                                    _ptr(dbias), _stream(stream)))


def fp16_conv_bn_workspace_bytes(conv: ConvDesc, bn: BnDesc) -> int:
    return int(lib().fp16_conv_bn_workspace_bytes(ctypes.byref(conv), ctypes.byref(bn)))


def fp16_conv_bn_relu_fwd(conv, bn, x, w, gamma, beta, residual, y, z, stats, ws=None,
                          ws_bytes=None, stream=None) -> None:
    _check("fp16_conv_bn_relu_fwd", lib().fp16_conv_bn_relu_fwd(
        ctypes.byref(conv), ctypes.byref(bn), _ptr(x), _ptr(w), _ptr(gamma), _ptr(beta),
        _ptr(residual), _ptr(y), _ptr(z), _ptr(stats), _ptr(ws), _wsb(ws, ws_bytes),
        _stream(stream)))


def fp16_conv_bn_relu_fwd_m(conv, bn, x, w, gamma, beta, residual, y, z, stats, mask, ws=None,
                            ws_bytes=None, stream=None) -> None:
    _check("fp16_conv_bn_relu_fwd_m", lib().fp16_conv_bn_relu_fwd_m(
        ctypes.byref(conv), ctypes.byref(bn), _ptr(x), _ptr(w), _ptr(gamma), _ptr(beta),
        _ptr(residual), _ptr(y), _ptr(z), _ptr(stats), _ptr(mask), _ptr(ws), _wsb(ws, ws_bytes),
        _stream(stream)))


def _wsb(ws, ws_bytes):
    if ws_bytes is not None:
        return int(ws_bytes)
    if ws is None or isinstance(ws, int):
        return 0
    return ws.numel() * ws.element_size()


# ---- conveniences that allocate outputs and workspaces with torch -----------

def workspace(nbytes: int, device="cuda"):
    import torch
    return torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)
