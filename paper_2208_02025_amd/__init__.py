"""Python binding of the gfx950 derived-operator library (libollie.so, include/ollie.h).

Argument marshalling only: every step of every operator runs in the library's HIP
kernels.  torch provides device memory and the current HIP stream.  There is no CPU
fallback: a missing libollie.so, or one built from sources other than those on disk
(its build digest differs), is built from csrc/ with hipcc on first use (and the call
raises if that fails), and tensors that are not on a GPU raise.

Layouts (contiguous):
  x   [n][h][w][c] (NHWC)          wt  [r][s][k][c]  (torch conv2d weight .permute(2,3,0,1),
                                                     conv_transpose2d weight .permute(2,3,1,0))
  out [n][ho][wo][k]
  q, k, v, o [b][l][d]             s   [b][l][2w+1]
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_DEFAULT_LIB = os.path.join(_HERE, "libollie.so")
# OLLIE_LIBRARY names another build of the library to load (the sanitizer test runs the
# host-side checks against an AddressSanitizer/UBSan build this way)
LIB_PATH = os.environ.get("OLLIE_LIBRARY") or _DEFAULT_LIB

OK, EINVAL, EDTYPE, EWORKSPACE, EALIGN, EHIP = range(6)
F32, BF16 = 0, 1
FUSE_EPILOGUE = 1 << 0
Y_BF16 = 1 << 1
BAND_STAGED = 1 << 2
BAND_MASK_INVALID = 1 << 3
DILATED_RESIDUES = 1 << 4
CONV_SPLIT_3X3 = 1 << 5


def FUSED_TILE(n: int) -> int:
    """Flag bits forcing tile shape n (0..14) of the fused convolution kernel."""
    return ((n + 1) & 0xff) << 16


def GEMM_TILE(n: int) -> int:
    """Flag bits forcing tile shape n (0..4) of the GEMM stage kernel."""
    return ((n + 1) & 0xf) << 24


def BAND_SHAPE(n: int) -> int:
    """Flag bits forcing wave shape n (0..3) of the fused band kernel."""
    return ((n + 1) & 0xff) << 16


_STATUS_NAMES = {OK: "OLLIE_OK", EINVAL: "OLLIE_EINVAL", EDTYPE: "OLLIE_EDTYPE",
                 EWORKSPACE: "OLLIE_EWORKSPACE", EALIGN: "OLLIE_EALIGN", EHIP: "OLLIE_EHIP"}

EXPORTS = ("derived_conv2d", "derived_dilated_conv2d", "derived_conv_transpose2d", "banded_bmm",
           "ollie_derived_conv2d_ex", "ollie_derived_dilated_conv2d_ex",
           "ollie_derived_conv_transpose2d_ex",
           "ollie_conv_out_hw", "ollie_conv_workspace_bytes", "ollie_band_workspace_bytes",
           "ollie_last_error", "ollie_version", "ollie_gemm_nt", "ollie_eop_offset_sum",
           "ollie_eop_convt_gather", "ollie_band_g2bmm", "ollie_band_softmax", "ollie_band_gbmm",
           "ollie_derived_conv2d_noalloc")


class ConvDesc(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("c", ctypes.c_int64), ("h", ctypes.c_int64),
                ("w", ctypes.c_int64), ("k", ctypes.c_int64), ("r", ctypes.c_int64),
                ("s", ctypes.c_int64),
                ("stride_h", ctypes.c_int32), ("stride_w", ctypes.c_int32),
                ("pad_h", ctypes.c_int32), ("pad_w", ctypes.c_int32),
                ("dil_h", ctypes.c_int32), ("dil_w", ctypes.c_int32),
                ("out_pad_h", ctypes.c_int32), ("out_pad_w", ctypes.c_int32),
                ("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32)]


class ConvEpilogue(ctypes.Structure):
    _fields_ = [("bias", ctypes.c_void_p), ("residual", ctypes.c_void_p),
                ("bias_dtype", ctypes.c_int32), ("residual_dtype", ctypes.c_int32),
                ("relu", ctypes.c_int32)]


class BandDesc(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int64), ("l", ctypes.c_int64), ("d", ctypes.c_int64),
                ("w", ctypes.c_int64), ("dilation", ctypes.c_int32), ("scale", ctypes.c_float),
                ("in_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32)]


class OllieError(RuntimeError):
    def __init__(self, status: int, fn: str, msg: str):
        super().__init__(f"{fn}: {_STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libollie.so, building it first if it is missing or was built from other
    sources than those now in csrc/ (its recorded build digest differs)."""
    global _lib
    if _lib is not None:
        return _lib
    from . import _build
    if path == _DEFAULT_LIB and not _build.is_current():
        _build.build()
    lib = ctypes.CDLL(path)
    p, i64, i32, u32, sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32,
                            ctypes.c_size_t)
    cdp, bdp = ctypes.POINTER(ConvDesc), ctypes.POINTER(BandDesc)
    edp = ctypes.POINTER(ConvEpilogue)
    sig = {
        "derived_conv2d": ([cdp, p, p, p, p, sz, u32, p], ctypes.c_int),
        "derived_dilated_conv2d": ([cdp, p, p, p, p, sz, u32, p], ctypes.c_int),
        "derived_conv_transpose2d": ([cdp, p, p, p, p, sz, u32, p], ctypes.c_int),
        "ollie_derived_conv2d_ex": ([cdp, p, p, p, p, sz, u32, edp, p], ctypes.c_int),
        "ollie_derived_dilated_conv2d_ex": ([cdp, p, p, p, p, sz, u32, edp, p], ctypes.c_int),
        "ollie_derived_conv_transpose2d_ex": ([cdp, p, p, p, p, sz, u32, edp, p], ctypes.c_int),
        "banded_bmm": ([bdp, p, p, p, p, p, p, sz, u32, p], ctypes.c_int),
        "ollie_derived_conv2d_noalloc": ([cdp, p, p, p, u32, p], ctypes.c_int),
        "ollie_conv_out_hw": ([cdp, ctypes.c_int, ctypes.POINTER(i64), ctypes.POINTER(i64)],
                              ctypes.c_int),
        "ollie_conv_workspace_bytes": ([cdp, ctypes.c_int, u32], sz),
        "ollie_band_workspace_bytes": ([bdp, u32], sz),
        "ollie_last_error": ([], ctypes.c_char_p),
        "ollie_version": ([], ctypes.c_char_p),
        "ollie_gemm_nt": ([i64, i64, i64, p, p, p, i32, i32, p], ctypes.c_int),
        "ollie_eop_offset_sum": ([cdp, p, i32, p, p], ctypes.c_int),
        "ollie_eop_convt_gather": ([cdp, p, i32, p, p], ctypes.c_int),
        "ollie_band_g2bmm": ([bdp, p, p, p, p], ctypes.c_int),
        "ollie_band_softmax": ([bdp, p, p, u32, p], ctypes.c_int),
        "ollie_band_gbmm": ([bdp, p, p, p, p], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(status: int, fn: str):
    if status != OK:
        raise OllieError(status, fn, load_library().ollie_last_error().decode())


def _pair(v):
    return (int(v), int(v)) if isinstance(v, int) else (int(v[0]), int(v[1]))


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.float32:
        return F32
    if dt == torch.bfloat16:
        return BF16
    raise ValueError(f"unsupported dtype {dt}; use torch.float32 or torch.bfloat16")


def _torch_dtype(code: int) -> torch.dtype:
    return torch.bfloat16 if code == BF16 else torch.float32


def _gpu(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor (the library has no CPU path)")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(dev) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def conv_desc(x_shape, wt_shape, stride=1, padding=0, dilation=1, output_padding=0,
              in_dtype=torch.bfloat16, out_dtype=torch.float32) -> ConvDesc:
    n, h, w, c = x_shape
    r, s, k, c2 = wt_shape
    if c != c2:
        raise ValueError(f"x has {c} channels but wt expects {c2}")
    (sh, sw), (ph, pw), (dh, dw), (oh, ow) = (_pair(stride), _pair(padding), _pair(dilation),
                                              _pair(output_padding))
    return ConvDesc(n, c, h, w, k, r, s, sh, sw, ph, pw, dh, dw, oh, ow,
                    _dtype_code(in_dtype), _dtype_code(out_dtype))


def conv_out_hw(desc: ConvDesc, transposed: bool):
    ho, wo = ctypes.c_int64(), ctypes.c_int64()
    _check(load_library().ollie_conv_out_hw(ctypes.byref(desc), int(transposed),
                                            ctypes.byref(ho), ctypes.byref(wo)),
           "ollie_conv_out_hw")
    return ho.value, wo.value


def conv_workspace_bytes(desc: ConvDesc, transposed: bool, flags: int = 0) -> int:
    return int(load_library().ollie_conv_workspace_bytes(ctypes.byref(desc), int(transposed),
                                                         flags))


def conv_epilogue(bias=None, residual=None, relu=False):
    """The element-wise tail act(conv + bias[k] + residual) as the library's struct, or
    None when there is no term (bias [K], residual shaped like out, fp32 or bf16)."""
    if bias is None and residual is None and not relu:
        return None
    for t, name in ((bias, "bias"), (residual, "residual")):
        if t is not None:
            _gpu(t, name)
    return ConvEpilogue(None if bias is None else bias.data_ptr(),
                        None if residual is None else residual.data_ptr(),
                        F32 if bias is None else _dtype_code(bias.dtype),
                        F32 if residual is None else _dtype_code(residual.dtype), int(bool(relu)))


def _conv(entry: str, transposed: bool, x, wt, stride, padding, dilation, output_padding,
          out_dtype, y_bf16, out, ws, fuse=False, bias=None, residual=None, relu=False,
          extra_flags=0):
    _gpu(x, "x")
    _gpu(wt, "wt")
    if x.dtype != wt.dtype:
        raise ValueError("x and wt must have the same dtype")
    desc = conv_desc(tuple(x.shape), tuple(wt.shape), stride, padding, dilation, output_padding,
                     x.dtype, out_dtype)
    flags = (Y_BF16 if y_bf16 else 0) | (FUSE_EPILOGUE if fuse else 0) | extra_flags
    ho, wo = conv_out_hw(desc, transposed)
    if out is None:
        out = torch.empty((desc.n, ho, wo, desc.k), dtype=out_dtype, device=x.device)
    else:
        _gpu(out, "out")
        if tuple(out.shape) != (desc.n, ho, wo, desc.k) or out.dtype != out_dtype:
            raise ValueError("out has the wrong shape or dtype")
    need = conv_workspace_bytes(desc, transposed, flags)
    if ws is None and need:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    epi = conv_epilogue(bias, residual, relu)
    if bias is not None and tuple(bias.shape) != (desc.k,):
        raise ValueError(f"bias must have shape ({desc.k},)")
    if residual is not None and tuple(residual.shape) != (desc.n, ho, wo, desc.k):
        raise ValueError("residual must have the shape of out")
    lib = load_library()
    if epi is None:
        st = getattr(lib, entry)(ctypes.byref(desc), _ptr(x), _ptr(wt), _ptr(out), _ptr(ws),
                                 ws_bytes, flags, _stream(x.device))
    else:
        entry = "ollie_" + entry + "_ex"
        st = getattr(lib, entry)(ctypes.byref(desc), _ptr(x), _ptr(wt), _ptr(out), _ptr(ws),
                                 ws_bytes, flags, ctypes.byref(epi), _stream(x.device))
    _check(st, entry)
    return out


def derived_conv2d(x, wt, stride=1, padding=0, out_dtype=torch.float32, y_bf16=False,
                   out=None, ws=None, fuse=False, bias=None, residual=None, relu=False,
                   split3x3=False, flags=0):
    """Conv2d (dilation 1) as GEMM + OffsetAdd eOperator (fuse=True: the fused
    expression, no Y).  x [N,H,W,C], wt [R,S,K,C].  bias / residual / relu: an
    element-wise tail act(conv + bias + residual) evaluated in the last kernel.
    split3x3=True (stride 1): the R x S kernel as ceil(R/3) x ceil(S/3) blocks of a 3x3
    convolution (fused by `fuse` where covered) whose partial outputs an OffsetAdd with
    offset step 3 sums (the Conv5x5 -> Conv3x3 derived form).  flags: extra flag bits
    (e.g. FUSED_TILE(n) / GEMM_TILE(n) tile overrides)."""
    return _conv("derived_conv2d", False, x, wt, stride, padding, 1, 0, out_dtype, y_bf16,
                 out, ws, fuse, bias, residual, relu,
                 (CONV_SPLIT_3X3 if split3x3 else 0) | flags)


NOALLOC_SCRATCH_BYTES = 64 << 20


def derived_conv2d_noalloc(x, wt, stride=1, padding=0, out_dtype=torch.float32, y_bf16=False,
                           out=None, fuse=False, split3x3=False, flags=0):
    """derived_conv2d through ollie_derived_conv2d_noalloc: the workspace is the library's
    static per-GPU scratch array (at most NOALLOC_SCRATCH_BYTES), so the library call
    itself allocates nothing.  `out` is allocated here when not given."""
    _gpu(x, "x")
    _gpu(wt, "wt")
    if x.dtype != wt.dtype:
        raise ValueError("x and wt must have the same dtype")
    desc = conv_desc(tuple(x.shape), tuple(wt.shape), stride, padding, 1, 0, x.dtype, out_dtype)
    fl = (Y_BF16 if y_bf16 else 0) | (FUSE_EPILOGUE if fuse else 0) | \
        (CONV_SPLIT_3X3 if split3x3 else 0) | flags
    ho, wo = conv_out_hw(desc, False)
    if out is None:
        out = torch.empty((desc.n, ho, wo, desc.k), dtype=out_dtype, device=x.device)
    else:
        _gpu(out, "out")
        if tuple(out.shape) != (desc.n, ho, wo, desc.k) or out.dtype != out_dtype:
            raise ValueError("out has the wrong shape or dtype")
    st = load_library().ollie_derived_conv2d_noalloc(ctypes.byref(desc), _ptr(x), _ptr(wt),
                                                     _ptr(out), fl, _stream(x.device))
    _check(st, "ollie_derived_conv2d_noalloc")
    return out


def derived_dilated_conv2d(x, wt, stride=1, padding=0, dilation=1, out_dtype=torch.float32,
                           y_bf16=False, out=None, ws=None, fuse=False, bias=None,
                           residual=None, relu=False, residues=False, flags=0):
    """Dilated Conv2d as GEMM + dilated OffsetAdd eOperator.  residues=True (implies
    fuse=True) evaluates it as dil_h*dil_w non-dilated convolutions over the residue
    sub-images of the input instead (stride 1).  flags: extra flag bits."""
    return _conv("derived_dilated_conv2d", False, x, wt, stride, padding, dilation, 0,
                 out_dtype, y_bf16, out, ws, fuse or residues, bias, residual, relu,
                 (DILATED_RESIDUES if residues else 0) | flags)


def derived_conv_transpose2d(x, wt, stride=1, padding=0, output_padding=0, dilation=1,
                             out_dtype=torch.float32, y_bf16=False, out=None, ws=None,
                             fuse=False, bias=None, residual=None, relu=False, flags=0):
    """ConvTranspose2d as GEMM on the unpadded input + selective-add eOperator.
    x [N,H,W,C_in], wt [R,S,C_out,C_in].  flags: extra flag bits."""
    return _conv("derived_conv_transpose2d", True, x, wt, stride, padding, dilation,
                 output_padding, out_dtype, y_bf16, out, ws, fuse, bias, residual, relu, flags)


def band_desc(q_shape, w, dilation, scale=1.0, out_dtype=torch.float32) -> BandDesc:
    b, l, d = q_shape
    return BandDesc(b, l, d, int(w), int(dilation), float(scale), BF16, _dtype_code(out_dtype))


def band_workspace_bytes(desc: BandDesc, flags: int) -> int:
    return int(load_library().ollie_band_workspace_bytes(ctypes.byref(desc), flags))


def banded_bmm(q, k, v, w, dilation=1, scale=1.0, mask_invalid=False, staged=False,
               out_dtype=torch.float32, return_s=False, out=None, ws=None, s_out=None,
               flags=0):
    """Banded dilated batched matmul + softmax + band-times-dense (q, k, v [B,L,64] bf16).

    Returns O, or (O, S) when return_s (staged path only).  flags: extra flag bits
    (e.g. BAND_SHAPE(n))."""
    for t, name in ((q, "q"), (k, "k"), (v, "v")):
        _gpu(t, name)
        if t.dtype != torch.bfloat16:
            raise ValueError(f"{name} must be bfloat16")
        if t.shape != q.shape:
            raise ValueError("q, k, v must have the same shape")
    desc = band_desc(tuple(q.shape), w, dilation, scale, out_dtype)
    flags |= (BAND_STAGED if staged or return_s else 0) | (BAND_MASK_INVALID if mask_invalid else 0)
    if out is None:
        out = torch.empty(tuple(q.shape), dtype=out_dtype, device=q.device)
    if return_s and s_out is None:
        s_out = torch.empty((desc.b, desc.l, 2 * desc.w + 1), dtype=torch.float32, device=q.device)
    need = band_workspace_bytes(desc, flags)
    if ws is None and need:
        ws = torch.empty(need, dtype=torch.uint8, device=q.device)
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    st = load_library().banded_bmm(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                   _ptr(s_out), _ptr(ws), ws_bytes, flags, _stream(q.device))
    _check(st, "banded_bmm")
    return (out, s_out) if return_s else out


# ------------------------------------------------------------------ stage entry points

def gemm_nt(a, b, y_dtype=torch.float32, out=None):
    """Y[m][n] = sum_k A[m][k] B[n][k] on the GEMM-stage kernel."""
    _gpu(a, "a")
    _gpu(b, "b")
    m, kk = a.shape
    n, kk2 = b.shape
    if kk != kk2 or a.dtype != b.dtype:
        raise ValueError("a and b must share k and dtype")
    if out is None:
        out = torch.empty((m, n), dtype=y_dtype, device=a.device)
    st = load_library().ollie_gemm_nt(m, n, kk, _ptr(a), _ptr(b), _ptr(out), _dtype_code(a.dtype),
                                      _dtype_code(out.dtype), _stream(a.device))
    _check(st, "ollie_gemm_nt")
    return out


def eop_gather(desc: ConvDesc, transposed: bool, y, out=None):
    """eOperator stage alone on a GEMM-stage scope y [n*h*w][r*s*k]."""
    _gpu(y, "y")
    ho, wo = conv_out_hw(desc, transposed)
    if out is None:
        out = torch.empty((desc.n, ho, wo, desc.k), dtype=_torch_dtype(desc.out_dtype),
                          device=y.device)
    entry = "ollie_eop_convt_gather" if transposed else "ollie_eop_offset_sum"
    st = getattr(load_library(), entry)(ctypes.byref(desc), _ptr(y), _dtype_code(y.dtype),
                                        _ptr(out), _stream(y.device))
    _check(st, entry)
    return out


def band_g2bmm(q, k, w, dilation=1, scale=1.0, s=None):
    desc = band_desc(tuple(q.shape), w, dilation, scale)
    if s is None:
        s = torch.empty((desc.b, desc.l, 2 * desc.w + 1), dtype=torch.float32, device=q.device)
    _check(load_library().ollie_band_g2bmm(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(s),
                                           _stream(q.device)), "ollie_band_g2bmm")
    return s


def band_softmax(s, w, dilation=1, mask_invalid=False, p=None):
    b, l, nb = s.shape
    desc = band_desc((b, l, 64), w, dilation)
    if p is None:
        p = torch.empty((b, l, nb), dtype=torch.bfloat16, device=s.device)
    _check(load_library().ollie_band_softmax(ctypes.byref(desc), _ptr(s), _ptr(p),
                                             BAND_MASK_INVALID if mask_invalid else 0,
                                             _stream(s.device)), "ollie_band_softmax")
    return p


def band_gbmm(p, v, w, dilation=1, out_dtype=torch.float32, o=None):
    desc = band_desc(tuple(v.shape), w, dilation, 1.0, out_dtype)
    if o is None:
        o = torch.empty(tuple(v.shape), dtype=out_dtype, device=v.device)
    _check(load_library().ollie_band_gbmm(ctypes.byref(desc), _ptr(p), _ptr(v), _ptr(o),
                                          _stream(v.device)), "ollie_band_gbmm")
    return o


def version() -> str:
    return load_library().ollie_version().decode()
