"""CPU oracle for the derived-operator path.  TEST INFRASTRUCTURE ONLY.

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import this
package; the product library never does, and this package never imports it.

``oracle.c`` (loaded through ctypes) evaluates every operator as its plain
nested-summation definition with double accumulation; ``derived_form.py`` is a
second, independent NumPy evaluation of the derived GEMM + eOperator form.

Tensors passed in are torch CPU tensors or NumPy arrays in the layouts described
in oracle.c; they are widened to float32 (exact for bf16) before the call.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import derived_form  # noqa: F401  (re-exported)

_HERE = os.path.dirname(os.path.abspath(__file__))
# OLLIE_ORACLE_LIBRARY names another build of oracle.c to load (the sanitizer test runs
# the pins against an AddressSanitizer/UBSan build this way)
_LIB_PATH = os.environ.get("OLLIE_ORACLE_LIBRARY") or os.path.join(_HERE, "liboracle.so")
_lib = None


class Geom(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int64) for name in
                ("n", "c", "h", "w", "k", "r", "s", "sh", "sw", "ph", "pw", "dh", "dw",
                 "oph", "opw")]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    p = ctypes.c_void_p
    i64 = ctypes.c_int64
    lib.oracle_threads.restype = ctypes.c_int
    lib.oracle_conv_out_size.restype = i64
    lib.oracle_conv_out_size.argtypes = [i64, i64, i64, i64, i64, i64, ctypes.c_int]
    for name in ("oracle_conv2d", "oracle_conv_transpose2d"):
        getattr(lib, name).argtypes = [ctypes.POINTER(Geom), p, p, p]
        getattr(lib, name).restype = None
    for name in ("oracle_conv2d_at", "oracle_conv_transpose2d_at"):
        getattr(lib, name).argtypes = [ctypes.POINTER(Geom), p, p, i64, p, p]
        getattr(lib, name).restype = None
    lib.oracle_band.argtypes = [i64, i64, i64, i64, i64, ctypes.c_double, ctypes.c_int,
                                p, p, p, i64, p, p, p, p]
    lib.oracle_band.restype = None
    _lib = lib
    return lib


def threads() -> int:
    return int(_load().oracle_threads())


def _f32(t) -> np.ndarray:
    if hasattr(t, "detach"):
        t = t.detach().cpu().float().numpy()
    return np.ascontiguousarray(np.asarray(t, dtype=np.float32))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _pair(v):
    return (v, v) if isinstance(v, int) else tuple(v)


def _geom(x, wt, stride, pad, dil, out_pad):
    n, h, w, c = x.shape
    r, s, k, c2 = wt.shape
    if c != c2:
        raise ValueError("channel mismatch between X and Wt")
    (sh, sw), (ph, pw), (dh, dw), (oph, opw) = (_pair(stride), _pair(pad), _pair(dil),
                                                _pair(out_pad))
    return Geom(n, c, h, w, k, r, s, sh, sw, ph, pw, dh, dw, oph, opw)


def conv_out_size(n_in, r, stride, pad, dil, out_pad=0, transposed=False) -> int:
    return int(_load().oracle_conv_out_size(n_in, r, stride, pad, dil, out_pad,
                                            1 if transposed else 0))


def _out_shape(g: Geom, transposed: bool):
    ho = conv_out_size(g.h, g.r, g.sh, g.ph, g.dh, g.oph, transposed)
    wo = conv_out_size(g.w, g.s, g.sw, g.pw, g.dw, g.opw, transposed)
    return (g.n, ho, wo, g.k)


def _conv(x, wt, stride, pad, dil, out_pad, transposed, idx):
    lib = _load()
    xa, wa = _f32(x), _f32(wt)
    g = _geom(xa, wa, stride, pad, dil, out_pad)
    shape = _out_shape(g, transposed)
    if idx is None:
        out = np.zeros(shape, dtype=np.float64)
        if out.size:
            fn = lib.oracle_conv_transpose2d if transposed else lib.oracle_conv2d
            fn(ctypes.byref(g), _ptr(xa), _ptr(wa), _ptr(out))
        return out
    ia = np.ascontiguousarray(np.asarray(idx, dtype=np.int64))
    vals = np.zeros(ia.shape[0], dtype=np.float64)
    fn = lib.oracle_conv_transpose2d_at if transposed else lib.oracle_conv2d_at
    fn(ctypes.byref(g), _ptr(xa), _ptr(wa), ia.shape[0], _ptr(ia), _ptr(vals))
    return vals


def conv2d(x, wt, stride=1, pad=0, dil=1, idx=None):
    """Convolution (cross-correlation) with stride, zero padding and dilation.

    x: [N,H,W,C], wt: [R,S,K,C] -> out [N,Ho,Wo,K] float64; with ``idx`` (flat
    indices into out) only those elements are evaluated and returned as a 1-D array."""
    return _conv(x, wt, stride, pad, dil, 0, False, idx)


def conv_transpose2d(x, wt, stride=1, pad=0, dil=1, out_pad=0, idx=None):
    """Transposed convolution (the adjoint of conv2d) in gather form; weight [R,S,K,C]
    maps C input channels to K output channels."""
    return _conv(x, wt, stride, pad, dil, out_pad, True, idx)


def conv_epilogue(conv, bias=None, residual=None, relu=False):
    """Element-wise tail of a convolution (section 6.3: OffsetAdd fused with the
    element-wise operators after it), by its definition in float64:
        out[n][ho][wo][k] = act(conv[n][ho][wo][k] + bias[k] + residual[n][ho][wo][k])
    with act = max(., 0) when relu, the identity otherwise.  conv is the operator's
    output [N, HO, WO, K]; bias [K] and residual [N, HO, WO, K] are optional."""
    y = np.asarray(conv, dtype=np.float64).copy()
    if bias is not None:
        y = y + _f32(bias).astype(np.float64).reshape(1, 1, 1, -1)
    if residual is not None:
        y = y + _f32(residual).astype(np.float64)
    if relu:
        y = np.where(y < 0.0, 0.0, y)
    return y


def band(q, k, v, w, dil, scale=1.0, mask=False, rows=None, want_s=True, want_p=True):
    """Banded dilated batched matmul + row softmax + band-times-dense product.

    q,k,v: [B,L,d].  rows: flat row ids b*L+i (None = all rows).
    Returns (S, P, O) with S,P [nrows, 2w+1] (or None) and O [nrows, d], float64;
    for rows=None they are reshaped to [B, L, ...]."""
    lib = _load()
    qa, ka, va = _f32(q), _f32(k), _f32(v)
    b_n, l, d = qa.shape
    nb = 2 * w + 1
    if rows is None:
        ra = None
        nrows = b_n * l
    else:
        ra = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        nrows = ra.shape[0]
    s = np.zeros((nrows, nb)) if want_s else None
    p = np.zeros((nrows, nb)) if want_p else None
    o = np.zeros((nrows, d))
    lib.oracle_band(b_n, l, d, w, dil, float(scale), 1 if mask else 0,
                    _ptr(qa), _ptr(ka), _ptr(va), nrows,
                    _ptr(ra) if ra is not None else None,
                    _ptr(s) if s is not None else None,
                    _ptr(p) if p is not None else None, _ptr(o))
    if rows is None:
        s = s.reshape(b_n, l, nb) if s is not None else None
        p = p.reshape(b_n, l, nb) if p is not None else None
        o = o.reshape(b_n, l, d)
    return s, p, o
