"""ctypes binding of ``libnmg.so`` (declared in ``include/nmg.h``).

Argument marshalling only: torch allocates the outputs on the input's device
and supplies the current HIP stream; every step of the computation runs in the
library's HIP kernels.  There is no fallback: if the library is missing or a
call fails, the binding raises.

Paper: STen (arXiv 2304.07613), Section 5 (n:m:g layout), 5.1 (sparse x dense
product), 5.2 (magnitude converter and conversion back to dense).
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

from . import build as _build

LIB_PATH = _build.LIB_PATH

F32, F16 = 0, 1
_DTYPE_CODE = {torch.float32: F32, torch.float16: F16}
KERNELS = {"auto": 0, "valu": 1, "mfma": 2, "mfma_general": 3, "mfma_scalar": 4, "mfma_f16": 5,
           "mfma_direct": 6, "smfmac_f16": 7, "valu_staged": 8, "mfma_wide": 9, "mfma_split": 10,
           "mfma_expand": 11}
_KERNEL_NAME = {v: k for k, v in KERNELS.items()}
EPILOGUES = {"none": 0, "gelu": 1, "add": 2}

OK, ERR_NULL, ERR_PARAM, ERR_SHAPE, ERR_DTYPE, ERR_ALIGN, ERR_LAUNCH, ERR_UNSUPPORTED, ERR_CAPACITY = \
    range(9)


class NmgError(RuntimeError):
    """A libnmg call returned a status other than NMG_OK."""

    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_str(status)} (status {status})")
        self.status = status


class _Layout(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int32), ("K", ctypes.c_int32), ("n", ctypes.c_int32),
                ("m", ctypes.c_int32), ("g", ctypes.c_int32), ("C", ctypes.c_int32),
                ("dtype", ctypes.c_int)]


class _PLayout(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int32), ("K", ctypes.c_int32), ("n", ctypes.c_int32),
                ("m", ctypes.c_int32), ("g", ctypes.c_int32), ("P", ctypes.c_int32),
                ("S", ctypes.c_int32), ("B", ctypes.c_int32), ("dtype", ctypes.c_int)]


_lib = None


def header_functions() -> list:
    """Names of the functions ``include/nmg.h`` declares."""
    with open(_build.HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^[A-Za-z_][\w \t\*]*?\b(nmg_\w+)\s*\(", text, re.M)))


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, lp = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.POINTER(_Layout)
    pp = ctypes.POINTER(_PLayout)
    sig = {
        "nmg_layout_init": ([lp, i32, i32, i32, i32, i32, ctypes.c_int], ctypes.c_int),
        "nmg_values_numel": ([lp], i64),
        "nmg_indices_numel": ([lp], i64),
        "nmg_compress": ([lp, vp, i64, vp, vp, vp], ctypes.c_int),
        "nmg_repack": ([lp, vp, i64, vp, vp, vp], ctypes.c_int),
        "nmg_spmm": ([lp, vp, vp, vp, i64, i64, vp, i64, vp], ctypes.c_int),
        "nmg_spmm_with": ([lp, ctypes.c_int, vp, vp, vp, i64, i64, vp, i64, vp], ctypes.c_int),
        "nmg_spmm_epilogue": ([lp, ctypes.c_int, ctypes.c_int, vp, vp, vp, i64, i64, vp, i64, vp,
                               i64, vp], ctypes.c_int),
        "nmg_spmm_epilogue_noalloc": ([lp, ctypes.c_int, ctypes.c_int, vp, vp, vp, i64, i64, vp,
                                       i64, vp, i64, vp], ctypes.c_int),
        "nmg_spmm_auto_kernel": ([lp, i64], ctypes.c_int),
        "nmg_densify": ([lp, vp, vp, vp, i64, vp], ctypes.c_int),
        "nmg_gelu": ([ctypes.c_int, vp, vp, i64, vp], ctypes.c_int),
        "nmg_add": ([ctypes.c_int, vp, vp, vp, i64, vp], ctypes.c_int),
        "nmg_p_layout_init": ([pp, i32, i32, i32, i32, i32, ctypes.c_int], ctypes.c_int),
        "nmg_p_compress": ([pp, vp, i64, vp, vp, vp], ctypes.c_int),
        "nmg_p_spmm": ([pp, vp, vp, vp, i64, i64, vp, i64, vp], ctypes.c_int),
        "nmg_p_spmm_with": ([pp, ctypes.c_int, vp, vp, vp, i64, i64, vp, i64, vp], ctypes.c_int),
        "nmg_p_refine": ([pp, vp, i64, vp, vp, vp], ctypes.c_int),
        "nmg_p_densify": ([pp, vp, vp, vp, i64, vp], ctypes.c_int),
        "nmg_x16_prepared_bytes": ([lp], i64),
        "nmg_x16_prepare": ([lp, vp, vp, vp, vp], ctypes.c_int),
        "nmg_spmm_x16": ([lp, vp, vp, i64, i64, vp, i64, vp], ctypes.c_int),
        "nmg_spmm_x16_epilogue": ([lp, vp, ctypes.c_int, vp, i64, i64, vp, i64, vp, i64, vp],
                                  ctypes.c_int),
        "nmg_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "nmg_version": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def status_str(status: int) -> str:
    return lib().nmg_status_str(status).decode()


def version() -> str:
    return lib().nmg_version().decode()


def _check(status: int, what: str):
    if status != OK:
        raise NmgError(status, what)


class Layout:
    """Shape of one n:m:g weight (``nmg_layout``)."""

    def __init__(self, M: int, K: int, n: int, m: int, g: int, dtype=torch.float32):
        if dtype not in _DTYPE_CODE:
            raise TypeError(f"unsupported dtype {dtype}")
        self.c = _Layout()
        _check(lib().nmg_layout_init(ctypes.byref(self.c), M, K, n, m, g, _DTYPE_CODE[dtype]),
               "nmg_layout_init")
        self.dtype = dtype

    M = property(lambda s: s.c.M)
    K = property(lambda s: s.c.K)
    n = property(lambda s: s.c.n)
    m = property(lambda s: s.c.m)
    g = property(lambda s: s.c.g)
    C = property(lambda s: s.c.C)

    @property
    def values_shape(self):
        return (self.M, self.C * self.n)

    @property
    def indices_shape(self):
        return (self.M // self.g, self.C * self.n)

    def __repr__(self):
        return (f"Layout(M={self.M}, K={self.K}, n={self.n}, m={self.m}, g={self.g}, "
                f"C={self.C}, dtype={self.dtype})")


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ptr(t: torch.Tensor):
    return ctypes.c_void_p(t.data_ptr())


def _need_cuda(*ts):
    """Every tensor on the current GPU: the library launches on the current
    HIP device, on that device's current stream."""
    cur = None
    for t in ts:
        if not t.is_cuda:
            raise ValueError("libnmg works on GPU tensors only")
        if cur is None:
            cur = torch.cuda.current_device()
        if t.device.index != cur:
            raise ValueError(f"tensor on {t.device}, but the current device is cuda:{cur} "
                             "(select it with torch.cuda.device)")


def _rows(t: torch.Tensor, name: str):
    """Leading dimension of a 2-D row-major tensor (unit stride along rows)."""
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D tensor with unit column stride")
    return t.stride(0)


def compress_into(layout: Layout, W: torch.Tensor, values: torch.Tensor, indices: torch.Tensor):
    """``nmg_compress`` into caller-allocated ``values`` / ``indices``."""
    _need_cuda(W, values, indices)
    if W.dtype != layout.dtype or values.dtype != layout.dtype or indices.dtype != torch.uint8:
        raise TypeError("dtype mismatch")
    if tuple(W.shape) != (layout.M, layout.K):
        raise ValueError(f"W must be {layout.M} x {layout.K}")
    if tuple(values.shape) != layout.values_shape or not values.is_contiguous():
        raise ValueError(f"values must be contiguous {layout.values_shape}")
    if tuple(indices.shape) != layout.indices_shape or not indices.is_contiguous():
        raise ValueError(f"indices must be contiguous {layout.indices_shape}")
    _check(lib().nmg_compress(ctypes.byref(layout.c), _ptr(W), _rows(W, "W"), _ptr(values),
                              _ptr(indices), _stream(W)), "nmg_compress")


def compress(W: torch.Tensor, n: int, m: int, g: int):
    """Dense W (M x K, GPU) -> (values, indices, layout)."""
    layout = Layout(W.shape[0], W.shape[1], n, m, g, W.dtype)
    values = torch.empty(layout.values_shape, dtype=W.dtype, device=W.device)
    indices = torch.empty(layout.indices_shape, dtype=torch.uint8, device=W.device)
    compress_into(layout, W, values, indices)
    return values, indices, layout


def repack(W: torch.Tensor, indices: torch.Tensor, layout: Layout) -> torch.Tensor:
    """Dense W (M x K, GPU) packed into the existing pattern `indices`
    (the fixed-mask path after a weight update) -> values."""
    _need_cuda(W, indices)
    if W.dtype != layout.dtype or indices.dtype != torch.uint8:
        raise TypeError("dtype mismatch")
    if tuple(W.shape) != (layout.M, layout.K):
        raise ValueError(f"W must be {layout.M} x {layout.K}")
    if tuple(indices.shape) != layout.indices_shape or not indices.is_contiguous():
        raise ValueError(f"indices must be contiguous {layout.indices_shape}")
    values = torch.empty(layout.values_shape, dtype=W.dtype, device=W.device)
    _check(lib().nmg_repack(ctypes.byref(layout.c), _ptr(W), _rows(W, "W"), _ptr(indices),
                            _ptr(values), _stream(W)), "nmg_repack")
    return values


# kernel families that run on prepared operands (made per call by
# nmg_spmm_with, or once by nmg_x16_prepare for nmg_spmm_x16), and the element
# type each takes
X16_KERNELS = {"mfma_wide": torch.float16, "mfma_split": torch.float32}


def x16_prepare(values, indices, layout: Layout) -> torch.Tensor:
    """``nmg_x16_prepare``: the prepared operands of a packed weight (bytes)."""
    _need_cuda(values, indices)
    nbytes = lib().nmg_x16_prepared_bytes(ctypes.byref(layout.c))
    if nbytes < 0:
        raise NmgError(ERR_UNSUPPORTED, "nmg_x16_prepared_bytes")
    prepared = torch.empty(int(nbytes), dtype=torch.uint8, device=values.device)
    _check(lib().nmg_x16_prepare(ctypes.byref(layout.c), _ptr(values), _ptr(indices),
                                 _ptr(prepared), _stream(values)), "nmg_x16_prepare")
    return prepared


def spmm_x16_into(layout: Layout, prepared, X, Y):
    """``nmg_spmm_x16`` into a caller-allocated Y (M x N)."""
    _need_cuda(prepared, X, Y)
    if X.dtype != layout.dtype or Y.dtype != layout.dtype:
        raise TypeError("dtype mismatch")
    if X.shape[0] != layout.K or Y.shape[0] != layout.M or Y.shape[1] != X.shape[1]:
        raise ValueError("X must be K x N and Y M x N")
    _check(lib().nmg_spmm_x16(ctypes.byref(layout.c), _ptr(prepared), _ptr(X), _rows(X, "X"),
                              X.shape[1], _ptr(Y), _rows(Y, "Y"), _stream(X)), "nmg_spmm_x16")


def spmm_x16_epilogue(layout: Layout, prepared, X, epilogue: str = "none", R=None, Y=None):
    """``nmg_spmm_x16_epilogue``: Y = W_s X ("none") or W_s X + R ("add") from
    prepared operands, the sum taken as the product is stored."""
    _need_cuda(prepared, X)
    if X.dtype != layout.dtype or X.shape[0] != layout.K:
        raise ValueError("X must be K x N of the layout's dtype")
    N = X.shape[1]
    if Y is None:
        Y = torch.empty((layout.M, N), dtype=X.dtype, device=X.device)
    _need_cuda(Y)
    if Y.dtype != layout.dtype or tuple(Y.shape) != (layout.M, N):
        raise ValueError("Y must be M x N of the layout's dtype")
    rp, ldr = ctypes.c_void_p(0), 0
    if epilogue == "add":
        if R is None:
            raise ValueError("the add epilogue needs R")
        _need_cuda(R)
        if R.dtype != layout.dtype or tuple(R.shape) != (layout.M, N):
            raise ValueError("R must be M x N of the layout's dtype")
        rp, ldr = _ptr(R), _rows(R, "R")
    _check(lib().nmg_spmm_x16_epilogue(ctypes.byref(layout.c), _ptr(prepared),
                                       EPILOGUES[epilogue], _ptr(X), _rows(X, "X"), N, rp, ldr,
                                       _ptr(Y), _rows(Y, "Y"), _stream(X)),
           "nmg_spmm_x16_epilogue")
    return Y


def spmm_into(layout: Layout, values, indices, X, Y, kernel: str = "auto"):
    """``nmg_spmm_with`` into a caller-allocated Y (M x N)."""
    _need_cuda(values, indices, X, Y)
    if X.dtype != layout.dtype or Y.dtype != layout.dtype or values.dtype != layout.dtype:
        raise TypeError("dtype mismatch")
    if X.shape[0] != layout.K or Y.shape[0] != layout.M or Y.shape[1] != X.shape[1]:
        raise ValueError("X must be K x N and Y M x N")
    if tuple(values.shape) != layout.values_shape or not values.is_contiguous():
        raise ValueError(f"values must be contiguous {layout.values_shape}")
    if tuple(indices.shape) != layout.indices_shape or not indices.is_contiguous():
        raise ValueError(f"indices must be contiguous {layout.indices_shape}")
    _check(lib().nmg_spmm_with(ctypes.byref(layout.c), KERNELS[kernel], _ptr(values),
                               _ptr(indices), _ptr(X), _rows(X, "X"), X.shape[1], _ptr(Y),
                               _rows(Y, "Y"), _stream(X)), "nmg_spmm")


def spmm(values, indices, X, layout: Layout, kernel: str = "auto"):
    """Y = W_s X for the packed weight (values, indices)."""
    Y = torch.empty((layout.M, X.shape[1]), dtype=X.dtype, device=X.device)
    spmm_into(layout, values, indices, X, Y, kernel)
    return Y


def spmm_epilogue(values, indices, X, layout: Layout, epilogue: str = "none", R=None,
                  kernel: str = "auto", Y=None):
    """Y = epilogue(W_s X): "none", "gelu" (GELU of the product) or "add"
    (product + R), bit for bit what spmm followed by gelu or add gives."""
    return _spmm_epilogue("nmg_spmm_epilogue", values, indices, X, layout, epilogue, R, kernel, Y)


def spmm_epilogue_noalloc(values, indices, X, layout: Layout, epilogue: str = "none", R=None,
                          kernel: str = "auto", Y=None):
    """``nmg_spmm_epilogue_noalloc``: spmm_epilogue without device allocation
    in the library (the prepared operands of mfma_wide / mfma_split go to the
    library's fixed per-GPU array; overlapping calls on one GPU race).  Y is
    allocated here when not given: pass Y to allocate nothing at all."""
    return _spmm_epilogue("nmg_spmm_epilogue_noalloc", values, indices, X, layout, epilogue, R,
                          kernel, Y)


def _spmm_epilogue(fn, values, indices, X, layout, epilogue, R, kernel, Y):
    _need_cuda(values, indices, X)
    if X.dtype != layout.dtype or values.dtype != layout.dtype:
        raise TypeError("dtype mismatch")
    if X.shape[0] != layout.K:
        raise ValueError("X must be K x N")
    if tuple(values.shape) != layout.values_shape or not values.is_contiguous():
        raise ValueError(f"values must be contiguous {layout.values_shape}")
    if tuple(indices.shape) != layout.indices_shape or not indices.is_contiguous():
        raise ValueError(f"indices must be contiguous {layout.indices_shape}")
    N = X.shape[1]
    if Y is None:
        Y = torch.empty((layout.M, N), dtype=X.dtype, device=X.device)
    _need_cuda(Y)
    if Y.dtype != layout.dtype or tuple(Y.shape) != (layout.M, N):
        raise ValueError("Y must be M x N of the layout's dtype")
    rp, ldr = ctypes.c_void_p(0), 0
    if epilogue == "add":
        if R is None:
            raise ValueError("the add epilogue needs R")
        _need_cuda(R)
        if R.dtype != layout.dtype or tuple(R.shape) != (layout.M, N):
            raise ValueError("R must be M x N of the layout's dtype")
        rp, ldr = _ptr(R), _rows(R, "R")
    _check(getattr(lib(), fn)(ctypes.byref(layout.c), KERNELS[kernel], EPILOGUES[epilogue],
                              _ptr(values), _ptr(indices), _ptr(X), _rows(X, "X"), N, rp, ldr,
                              _ptr(Y), _rows(Y, "Y"), _stream(X)), fn)
    return Y


def auto_kernel(layout: Layout, N: int) -> str:
    return _KERNEL_NAME[lib().nmg_spmm_auto_kernel(ctypes.byref(layout.c), N)]


def densify(values, indices, layout: Layout):
    """(values, indices) -> dense M x K weight (zeros at dropped positions)."""
    _need_cuda(values, indices)
    out = torch.empty((layout.M, layout.K), dtype=layout.dtype, device=values.device)
    _check(lib().nmg_densify(ctypes.byref(layout.c), _ptr(values), _ptr(indices), _ptr(out),
                             layout.K, _stream(values)), "nmg_densify")
    return out


def gelu(x: torch.Tensor, out: torch.Tensor | None = None):
    _need_cuda(x)
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    out = torch.empty_like(x) if out is None else out
    _check(lib().nmg_gelu(_DTYPE_CODE[x.dtype], _ptr(x), _ptr(out), x.numel(), _stream(x)),
           "nmg_gelu")
    return out


def add(a: torch.Tensor, b: torch.Tensor, out: torch.Tensor | None = None):
    _need_cuda(a, b)
    if a.shape != b.shape or a.dtype != b.dtype or not (a.is_contiguous() and b.is_contiguous()):
        raise ValueError("a and b must be contiguous tensors of one shape and dtype")
    out = torch.empty_like(a) if out is None else out
    _check(lib().nmg_add(_DTYPE_CODE[a.dtype], _ptr(a), _ptr(b), _ptr(out), a.numel(),
                         _stream(a)), "nmg_add")
    return out


# ------------------------------------------------ the paper's chunked layout

class PLayout:
    """Shape of one weight in the paper's chunked layout (``nmg_p_layout``)."""

    def __init__(self, M: int, K: int, n: int, m: int, g: int, dtype=torch.float32):
        if dtype not in _DTYPE_CODE:
            raise TypeError(f"unsupported dtype {dtype}")
        self.c = _PLayout()
        _check(lib().nmg_p_layout_init(ctypes.byref(self.c), M, K, n, m, g, _DTYPE_CODE[dtype]),
               "nmg_p_layout_init")
        self.dtype = dtype

    M = property(lambda s: s.c.M)
    K = property(lambda s: s.c.K)
    n = property(lambda s: s.c.n)
    m = property(lambda s: s.c.m)
    g = property(lambda s: s.c.g)
    P = property(lambda s: s.c.P)
    S = property(lambda s: s.c.S)
    B = property(lambda s: s.c.B)

    @property
    def values_shape(self):
        return (self.M, self.B * self.n)

    @property
    def index_shape(self):
        return (self.M, self.B)


def p_compress(W: torch.Tensor, n: int, m: int, g: int):
    """Dense W (M x K, GPU) -> (values, index, layout) in the chunked layout."""
    _need_cuda(W)
    layout = PLayout(W.shape[0], W.shape[1], n, m, g, W.dtype)
    values = torch.empty(layout.values_shape, dtype=W.dtype, device=W.device)
    index = torch.empty(layout.index_shape, dtype=torch.uint8, device=W.device)
    _check(lib().nmg_p_compress(ctypes.byref(layout.c), _ptr(W), _rows(W, "W"), _ptr(values),
                                _ptr(index), _stream(W)), "nmg_p_compress")
    return values, index, layout


def _p_check(layout: PLayout, values, index):
    _need_cuda(values, index)
    if values.dtype != layout.dtype or index.dtype != torch.uint8:
        raise TypeError("dtype mismatch")
    if tuple(values.shape) != layout.values_shape or not values.is_contiguous():
        raise ValueError(f"values must be contiguous {layout.values_shape}")
    if tuple(index.shape) != layout.index_shape or not index.is_contiguous():
        raise ValueError(f"index must be contiguous {layout.index_shape}")


def p_spmm(values, index, X, layout: PLayout, kernel: str = "auto"):
    """Y = W_s X for the chunked layout; kernel is "auto", "valu" or "mfma"."""
    _p_check(layout, values, index)
    _need_cuda(X)
    if X.dtype != layout.dtype or X.shape[0] != layout.K:
        raise ValueError("X must be K x N of the layout's dtype")
    if kernel not in ("auto", "valu", "mfma"):
        raise ValueError(f"unknown chunked-layout kernel {kernel!r}")
    Y = torch.empty((layout.M, X.shape[1]), dtype=X.dtype, device=X.device)
    _check(lib().nmg_p_spmm_with(ctypes.byref(layout.c), KERNELS[kernel], _ptr(values),
                                 _ptr(index), _ptr(X), _rows(X, "X"), X.shape[1], _ptr(Y),
                                 _rows(Y, "Y"), _stream(X)),
           "nmg_p_spmm_with")
    return Y


def p_densify(values, index, layout: PLayout):
    """Chunked layout -> dense M x K weight."""
    _p_check(layout, values, index)
    out = torch.empty((layout.M, layout.K), dtype=layout.dtype, device=values.device)
    _check(lib().nmg_p_densify(ctypes.byref(layout.c), _ptr(values), _ptr(index), _ptr(out),
                               layout.K, _stream(values)), "nmg_p_densify")
    return out


def p_refine(W: torch.Tensor, index: torch.Tensor, layout: PLayout):
    """The swap search of Section 5.2's GPU converter from the packing `index`:
    returns new (values, index); the inputs are not changed."""
    _need_cuda(W, index)
    if W.dtype != layout.dtype or index.dtype != torch.uint8:
        raise TypeError("dtype mismatch")
    if tuple(W.shape) != (layout.M, layout.K):
        raise ValueError(f"W must be {layout.M} x {layout.K}")
    if tuple(index.shape) != layout.index_shape:
        raise ValueError(f"index must be {layout.index_shape}")
    idx = index.contiguous().clone()
    values = torch.empty(layout.values_shape, dtype=W.dtype, device=W.device)
    _check(lib().nmg_p_refine(ctypes.byref(layout.c), _ptr(W), _rows(W, "W"), _ptr(values),
                              _ptr(idx), _stream(W)), "nmg_p_refine")
    return values, idx
