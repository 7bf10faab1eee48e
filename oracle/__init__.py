"""Python view of the CPU oracle -- TEST INFRASTRUCTURE ONLY.

The oracle (``fp16_oracle.cpp``) is the plain float64 definition of the
all-FP16 training hot path of arXiv:1911.07384 that the HIP kernels are
checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package; the product path
never does.

Arrays are numpy: binary16 tensors are passed as ``np.float16`` (or their
``uint16`` bit patterns) and returned as ``np.float16``.
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fp16_oracle.cpp")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(verbose: bool = False) -> str:
    """Compile the oracle with the host compiler (no GPU code involved)."""
    cmd = ["g++", "-O2", "-std=c++17", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-shared", "-fPIC", _SRC, "-o", _LIB + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_F32 = ctypes.c_float
_F64 = ctypes.c_double
_INT = ctypes.c_int

_SIGS = {
    "oracle_h2d": (_F64, [ctypes.c_uint16]),
    "oracle_rne16": (ctypes.c_uint16, [_F64]),
    "oracle_h2d_array": (None, [_P, _P, _I64]),
    "oracle_rne16_array": (None, [_P, _P, _I64]),
    "oracle_rne16_f32_array": (None, [_P, _P, _I64]),
    "oracle_num_threads": (_INT, []),
    "oracle_set_num_threads": (None, [_INT]),
    "oracle_conv_out_dims": (None, [_P, _P, _P]),
    "oracle_conv_fwd": (None, [_P, _P, _P, _P, _P]),
    "oracle_conv_dgrad": (None, [_P, _P, _P, _P, _P]),
    "oracle_conv_wgrad": (None, [_P, _P, _P, _P, _P]),
    "oracle_conv_dgrad_add": (None, [_P, _P, _P, _P, _P, _P]),
    "oracle_conv_fwd_at": (None, [_P, _P, _P, _P, _I64, _P]),
    "oracle_conv_dgrad_at": (None, [_P, _P, _P, _P, _I64, _P]),
    "oracle_conv_wgrad_at": (None, [_P, _P, _P, _P, _I64, _P]),
    "oracle_bn_fwd": (None, [_P, _P, _P, _P, _P, _F32, _F32, _INT, _P, _P, _P, _P, _INT]),
    "oracle_bn_apply_f32": (None, [_P, _P, _P, _P, _P, _P, _P, _F32, _INT, _P, _INT]),
    "oracle_bn_bwd": (None, [_P, _P, _P, _P, _P, _F32, _F32, _INT, _P, _P, _P, _P, _P, _P, _P,
                             _INT, _P]),
    "oracle_sgd_f32": (None, [_P, _P, _P, _I64, _F32, _F32, _F32]),
    "oracle_sgd_f64": (None, [_P, _P, _P, _I64, _F64, _F64, _F64]),
    "oracle_pool_out_dims": (None, [_P, _P, _P]),
    "oracle_maxpool_fwd": (None, [_P, _P, _P, _P]),
    "oracle_maxpool_bwd": (None, [_P, _P, _P, _P]),
    "oracle_avgpool_fwd": (None, [_P, _P, _P, _P]),
    "oracle_avgpool_bwd": (None, [_P, _P, _P]),
    "oracle_softmax_ce": (None, [_I64, _I64, _P, _P, _P, _P, _P, _P, _P]),
    "oracle_fma16": (ctypes.c_uint16, [ctypes.c_uint16, ctypes.c_uint16, ctypes.c_uint16]),
    "oracle_fma16_array": (None, [_P, _P, _P, _P, _I64]),
    "oracle_sgd_f16": (None, [_P, _P, _P, _I64, _F32, _F32, _F32]),
    "oracle_conv_fwd_f16acc": (None, [_P, _P, _P, _P]),
    "oracle_conv_dgrad_f16acc": (None, [_P, _P, _P, _P]),
    "oracle_conv_wgrad_f16acc": (None, [_P, _P, _P, _P]),
    "oracle_conv_fwd_f16acc_at": (None, [_P, _P, _P, _P, _I64, _P]),
    "oracle_conv_dgrad_f16acc_at": (None, [_P, _P, _P, _P, _I64, _P]),
    "oracle_conv_wgrad_f16acc_at": (None, [_P, _P, _P, _P, _I64, _P]),
}


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        l = ctypes.CDLL(_LIB)
        for name, (res, args) in _SIGS.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _h(a) -> np.ndarray:
    """Contiguous uint16 bit view of a binary16 array (float16 or uint16)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.float16:
        return a.view(np.uint16)
    assert a.dtype == np.uint16, a.dtype
    return a


def num_threads() -> int:
    return lib().oracle_num_threads()


def set_num_threads(n: int) -> None:
    """OpenMP threads of the following oracle calls (for single-core timing)."""
    lib().oracle_set_num_threads(int(n))


# ---- codec ----------------------------------------------------------------

def h2d(h) -> np.ndarray:
    h = _h(h)
    out = np.empty(h.shape, np.float64)
    lib().oracle_h2d_array(_ptr(h), _ptr(out), h.size)
    return out


def rne16(v) -> np.ndarray:
    """Round float64 (or float32) values to binary16, ties to even."""
    v = np.ascontiguousarray(v)
    out = np.empty(v.shape, np.uint16)
    if v.dtype == np.float32:
        lib().oracle_rne16_f32_array(_ptr(v), _ptr(out), v.size)
    else:
        v = np.ascontiguousarray(v, dtype=np.float64)
        lib().oracle_rne16_array(_ptr(v), _ptr(out), v.size)
    return out.view(np.float16)


# ---- convolution ----------------------------------------------------------

def conv_shape(n, c, h, w, k, r, s, stride=1, pad=0, layout="NHWC") -> np.ndarray:
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    lay = {"NHWC": 0, "NCHW": 1}[layout]
    return np.array([n, c, h, w, k, r, s, sh, sw, ph, pw, lay], dtype=np.int32)


def conv_out_dims(shp) -> tuple:
    p = np.zeros(1, np.int32)
    q = np.zeros(1, np.int32)
    lib().oracle_conv_out_dims(_ptr(shp), _ptr(p), _ptr(q))
    return int(p[0]), int(q[0])


def _act_shape(shp, which):
    n, c, h, w, k, r, s = (int(v) for v in shp[:7])
    lay = int(shp[11])
    p, q = conv_out_dims(shp)
    if which == "x":
        return (n, h, w, c) if lay == 0 else (n, c, h, w)
    if which == "y":
        return (n, p, q, k) if lay == 0 else (n, k, p, q)
    return (k, r, s, c) if lay == 0 else (k, c, r, s)


def conv_fwd(shp, x, w):
    """Returns (y64, y16): the float64 sums and their binary16 rounding."""
    x, w = _h(x), _h(w)
    ys = _act_shape(shp, "y")
    y64 = np.empty(ys, np.float64)
    y16 = np.empty(ys, np.uint16)
    lib().oracle_conv_fwd(_ptr(shp), _ptr(x), _ptr(w), _ptr(y64), _ptr(y16))
    return y64, y16.view(np.float16)


def conv_dgrad(shp, dy, w):
    dy, w = _h(dy), _h(w)
    xs = _act_shape(shp, "x")
    dx64 = np.empty(xs, np.float64)
    dx16 = np.empty(xs, np.uint16)
    lib().oracle_conv_dgrad(_ptr(shp), _ptr(dy), _ptr(w), _ptr(dx64), _ptr(dx16))
    return dx64, dx16.view(np.float16)


def conv_dgrad_add(shp, dy, w, addend):
    """Data gradient plus a binary16 addend, one rounding: (dx64, dx16)."""
    dy, w, addend = _h(dy), _h(w), _h(addend)
    xs = _act_shape(shp, "x")
    assert addend.shape == xs, (addend.shape, xs)
    dx64 = np.empty(xs, np.float64)
    dx16 = np.empty(xs, np.uint16)
    lib().oracle_conv_dgrad_add(_ptr(shp), _ptr(dy), _ptr(w), _ptr(addend), _ptr(dx64), _ptr(dx16))
    return dx64, dx16.view(np.float16)


def conv_wgrad(shp, x, dy):
    x, dy = _h(x), _h(dy)
    ws = _act_shape(shp, "w")
    dw64 = np.empty(ws, np.float64)
    dw16 = np.empty(ws, np.uint16)
    lib().oracle_conv_wgrad(_ptr(shp), _ptr(x), _ptr(dy), _ptr(dw64), _ptr(dw16))
    return dw64, dw16.view(np.float16)


def _at(fn, shp, a, b, idx):
    a, b = _h(a), _h(b)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.shape, np.float64)
    fn(_ptr(shp), _ptr(a), _ptr(b), _ptr(idx), idx.size, _ptr(out))
    return out


def conv_fwd_at(shp, x, w, idx):
    """float64 forward sums at flat output indices ``idx`` (output layout)."""
    return _at(lib().oracle_conv_fwd_at, shp, x, w, idx)


def conv_dgrad_at(shp, dy, w, idx):
    return _at(lib().oracle_conv_dgrad_at, shp, dy, w, idx)


def conv_wgrad_at(shp, x, dy, idx):
    return _at(lib().oracle_conv_wgrad_at, shp, x, dy, idx)


# ---- batch normalisation --------------------------------------------------

def bn_shape(n, c, h, w, layout="NHWC") -> np.ndarray:
    return np.array([n, c, h, w, {"NHWC": 0, "NCHW": 1}[layout]], dtype=np.int32)


def bn_fwd(shp, x, gamma, beta, residual=None, eps=1e-5, post_scale=1.0, relu=True, swap=False):
    """Returns dict(mean, var, y64, y) with y binary16.  swap: the BN swap
    (the shortcut joins before gamma; needs the residual)."""
    x, gamma, beta = _h(x), _h(gamma), _h(beta)
    res = None if residual is None else _h(residual)
    if swap and res is None:
        raise ValueError("the BN swap needs the residual")
    C = int(shp[1])
    mean = np.empty(C, np.float64)
    var = np.empty(C, np.float64)
    y64 = np.empty(x.shape, np.float64)
    y16 = np.empty(x.shape, np.uint16)
    lib().oracle_bn_fwd(_ptr(shp), _ptr(x), _ptr(gamma), _ptr(beta), _ptr(res),
                        float(eps), float(post_scale), int(bool(relu)),
                        _ptr(mean), _ptr(var), _ptr(y64), _ptr(y16), int(bool(swap)))
    return {"mean": mean, "var": var, "y64": y64, "y": y16.view(np.float16)}


def bn_apply_f32(shp, x, gamma, beta, mean, rstd, residual=None, post_scale=1.0, relu=True,
                 swap=False):
    """Declared float32 apply with given float32 statistics; binary16 result."""
    x, gamma, beta = _h(x), _h(gamma), _h(beta)
    res = None if residual is None else _h(residual)
    if swap and res is None:
        raise ValueError("the BN swap needs the residual")
    mean = np.ascontiguousarray(mean, dtype=np.float32)
    rstd = np.ascontiguousarray(rstd, dtype=np.float32)
    y16 = np.empty(x.shape, np.uint16)
    lib().oracle_bn_apply_f32(_ptr(shp), _ptr(x), _ptr(gamma), _ptr(beta), _ptr(res),
                              _ptr(mean), _ptr(rstd), float(post_scale), int(bool(relu)),
                              _ptr(y16), int(bool(swap)))
    return y16.view(np.float16)


def bn_bwd(shp, x, y, dy, gamma, eps=1e-5, post_scale=1.0, relu=True, want_dres=False,
           swap=False, residual=None):
    """Returns dict(dx, dgamma, dbeta, dres, dx64, dgamma64, dbeta64).  With
    swap the residual is needed (dgamma includes sum g*r)."""
    x, dy, gamma = _h(x), _h(dy), _h(gamma)
    y = None if y is None else _h(y)
    res = None if residual is None else _h(residual)
    if swap and res is None:
        raise ValueError("the BN swap needs the residual")
    if relu and y is None:
        raise ValueError("the ReLU mask needs the forward output y")
    C = int(shp[1])
    dx = np.empty(x.shape, np.uint16)
    dx64 = np.empty(x.shape, np.float64)
    dg = np.empty(C, np.uint16)
    db = np.empty(C, np.uint16)
    dg64 = np.empty(C, np.float64)
    db64 = np.empty(C, np.float64)
    dres = np.empty(x.shape, np.uint16) if want_dres else None
    lib().oracle_bn_bwd(_ptr(shp), _ptr(x), _ptr(y), _ptr(dy), _ptr(gamma), float(eps),
                        float(post_scale), int(bool(relu)), _ptr(dx), _ptr(dg), _ptr(db),
                        _ptr(dres), _ptr(dx64), _ptr(dg64), _ptr(db64), int(bool(swap)),
                        _ptr(res))
    return {"dx": dx.view(np.float16), "dgamma": dg.view(np.float16),
            "dbeta": db.view(np.float16),
            "dres": None if dres is None else dres.view(np.float16),
            "dx64": dx64, "dgamma64": dg64, "dbeta64": db64}


# ---- SGD ------------------------------------------------------------------

def sgd_f32(w, g, m, lr, momentum, weight_decay):
    """Declared float32 sequence; returns new (w, m) as binary16 copies."""
    w = _h(w).copy()
    m = _h(m).copy()
    g = _h(g)
    lib().oracle_sgd_f32(_ptr(w), _ptr(g), _ptr(m), w.size, float(lr), float(momentum),
                         float(weight_decay))
    return w.view(np.float16), m.view(np.float16)


def sgd_f64(w, g, m, lr, momentum, weight_decay):
    w = _h(w).copy()
    m = _h(m).copy()
    g = _h(g)
    lib().oracle_sgd_f64(_ptr(w), _ptr(g), _ptr(m), w.size, float(lr), float(momentum),
                         float(weight_decay))
    return w.view(np.float16), m.view(np.float16)


# ---- strict binary16 arithmetic (all operations in FP16) --------------------

def fma16(a, b, c):
    """Elementwise binary16 fused multiply-add, one rounding (arrays)."""
    a, b, c = (_h(np.asarray(v, dtype=np.float16) if np.asarray(v).dtype != np.uint16 else v)
               for v in (a, b, c))
    a, b, c = np.broadcast_arrays(a, b, c)
    a, b, c = (np.ascontiguousarray(v) for v in (a, b, c))
    out = np.empty(a.shape, np.uint16)
    lib().oracle_fma16_array(_ptr(a), _ptr(b), _ptr(c), _ptr(out), a.size)
    return out.view(np.float16)


def sgd_f16(w, g, m, lr, momentum, weight_decay):
    """SGD with every operation a binary16 fma; the scalars are the binary16
    roundings of the float32 arguments."""
    w = _h(w).copy()
    m = _h(m).copy()
    g = _h(g)
    lib().oracle_sgd_f16(_ptr(w), _ptr(g), _ptr(m), w.size, float(lr), float(momentum),
                         float(weight_decay))
    return w.view(np.float16), m.view(np.float16)


def _f16acc(fn, shp, a, b, which):
    a, b = _h(a), _h(b)
    out = np.empty(_act_shape(shp, which), np.uint16)
    fn(_ptr(shp), _ptr(a), _ptr(b), _ptr(out))
    return out.view(np.float16)


def conv_fwd_f16acc(shp, x, w):
    """Forward convolution with every operation in binary16: each output is
    a chain of binary16 fmas from +0 over its in-image terms, taps (r, s)
    row-major, channels ascending within a tap."""
    return _f16acc(lib().oracle_conv_fwd_f16acc, shp, x, w, "y")


def conv_dgrad_f16acc(shp, dy, w):
    """Data gradient as a binary16 fma chain: taps (r, s) row-major that
    reach the position from the output grid, output channels ascending."""
    return _f16acc(lib().oracle_conv_dgrad_f16acc, shp, dy, w, "x")


def conv_wgrad_f16acc(shp, x, dy):
    """Weight gradient as a binary16 fma chain over the output pixels
    (n, p, q) in order, in-image taps only."""
    return _f16acc(lib().oracle_conv_wgrad_f16acc, shp, x, dy, "w")


def _f16acc_at(fn, shp, a, b, idx):
    a, b = _h(a), _h(b)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, np.uint16)
    fn(_ptr(shp), _ptr(a), _ptr(b), _ptr(idx), idx.size, _ptr(out))
    return out.view(np.float16)


def conv_fwd_f16acc_at(shp, x, w, idx):
    """conv_fwd_f16acc at the flat output indices idx only."""
    return _f16acc_at(lib().oracle_conv_fwd_f16acc_at, shp, x, w, idx)


def conv_dgrad_f16acc_at(shp, dy, w, idx):
    return _f16acc_at(lib().oracle_conv_dgrad_f16acc_at, shp, dy, w, idx)


def conv_wgrad_f16acc_at(shp, x, dy, idx):
    return _f16acc_at(lib().oracle_conv_wgrad_f16acc_at, shp, x, dy, idx)


# ---- pooling, classifier bias and loss --------------------------------------

def pool_shape(n, c, h, w, r, s, stride=1, pad=0, layout="NHWC") -> np.ndarray:
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    return np.array([n, c, h, w, r, s, sh, sw, ph, pw, {"NHWC": 0, "NCHW": 1}[layout]],
                    dtype=np.int32)


def pool_out_dims(shp) -> tuple:
    p = np.zeros(1, np.int32)
    q = np.zeros(1, np.int32)
    lib().oracle_pool_out_dims(_ptr(shp), _ptr(p), _ptr(q))
    return int(p[0]), int(q[0])


def _pool_y_shape(shp):
    n, c = int(shp[0]), int(shp[1])
    p, q = pool_out_dims(shp)
    return (n, p, q, c) if int(shp[10]) == 0 else (n, c, p, q)


def maxpool_fwd(shp, x):
    """Returns (y, idx): binary16 maxima and the winning tap r*S+s (uint8)."""
    x = _h(x)
    ys = _pool_y_shape(shp)
    y = np.empty(ys, np.uint16)
    idx = np.empty(ys, np.uint8)
    lib().oracle_maxpool_fwd(_ptr(shp), _ptr(x), _ptr(y), _ptr(idx))
    return y.view(np.float16), idx


def maxpool_bwd(shp, x, dy):
    x, dy = _h(x), _h(dy)
    dx = np.empty(x.shape, np.uint16)
    lib().oracle_maxpool_bwd(_ptr(shp), _ptr(x), _ptr(dy), _ptr(dx))
    return dx.view(np.float16)


def avgpool_fwd(shp, x):
    """Global average pool: returns (y64, y16), each [N, C]."""
    x = _h(x)
    n, c = int(shp[0]), int(shp[1])
    y64 = np.empty((n, c), np.float64)
    y16 = np.empty((n, c), np.uint16)
    lib().oracle_avgpool_fwd(_ptr(shp), _ptr(x), _ptr(y64), _ptr(y16))
    return y64, y16.view(np.float16)


def avgpool_bwd(shp, dy):
    dy = _h(dy)
    n, c, h, w = (int(v) for v in shp[:4])
    xs = (n, h, w, c) if int(shp[10]) == 0 else (n, c, h, w)
    dx = np.empty(xs, np.uint16)
    lib().oracle_avgpool_bwd(_ptr(shp), _ptr(dy), _ptr(dx))
    return dx.view(np.float16)


def softmax_ce(z, b, labels):
    """Classifier bias + softmax cross-entropy, mean over the batch.

    Returns dict(loss (mean), loss_rows, dz, db); dz is the gradient of the
    mean loss with respect to z (and to the logits), db that of the bias."""
    z, b = _h(z), _h(b)
    n, k = z.shape
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    assert labels.shape == (n,) and b.shape == (k,)
    rows = np.empty(n, np.float64)
    mean = np.empty(1, np.float64)
    dz = np.empty((n, k), np.uint16)
    db = np.empty(k, np.uint16)
    lib().oracle_softmax_ce(n, k, _ptr(z), _ptr(b), _ptr(labels), _ptr(rows), _ptr(mean),
                            _ptr(dz), _ptr(db))
    return {"loss": float(mean[0]), "loss_rows": rows, "dz": dz.view(np.float16),
            "db": db.view(np.float16)}
