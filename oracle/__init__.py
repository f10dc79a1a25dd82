"""CPU oracle for the grouped n:m (n:m:g) layout.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
CPU-baseline leg of the benchmark may import this module; the GPU library never
does, and the two share no code.  The arithmetic lives in ``nmg_oracle.c``
(plain C, binary64 accumulation); this module only marshals NumPy arrays.

Paper: STen (arXiv 2304.07613), Section 5 (the n:m:g layout), Section 5.1 (the
sparse x dense product), Section 5.2 (the L1-maximising converter and the
conversion back to dense), Section 6.1 (the energy metric).

Functions with no independent pin: none.  Every entry point here is checked in
``tests/test_oracle.py`` against brute force, closed forms, special cases that
reduce to library routines, or hand-worked examples.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "nmg_oracle.c")
LIB_PATH = os.path.join(_HERE, "liboracle_nmg.so")

F32, F16 = 0, 1
_STATUS = {0: "ok", 1: "bad parameter", 2: "bad shape", 3: "bad indices"}


class OracleError(ValueError):
    """The oracle rejected its arguments (status code in ``.status``)."""

    def __init__(self, status: int, what: str):
        super().__init__(f"oracle {what}: {_STATUS.get(status, status)}")
        self.status = status


def build(force: bool = True) -> str:
    """Compile ``nmg_oracle.c`` with gcc into ``liboracle_nmg.so``.

    Plain -O2, no fast-math and no FMA contraction, so binary32 score sums are
    rounded after every addition as the selection rule requires.
    """
    if not force and os.path.exists(LIB_PATH):
        return LIB_PATH
    tmp = LIB_PATH + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fopenmp",
           "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH) or (
            os.path.getmtime(LIB_PATH) < os.path.getmtime(_SRC)):
        build()
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p
    lib.oracle_compress.argtypes = [i32, i64, i64, i32, i32, i32, vp, i64, vp, vp]
    lib.oracle_densify.argtypes = [i32, i64, i64, i32, i32, i32, vp, vp, vp, i64, vp]
    lib.oracle_repack.argtypes = [i32, i64, i64, i32, i32, i32, vp, i64, vp, vp]
    lib.oracle_p_patterns.argtypes = [i32, i32, vp]
    lib.oracle_p_compress.argtypes = [i32, i64, i64, i32, i32, i32, vp, i64, vp, vp]
    lib.oracle_p_densify.argtypes = [i32, i64, i64, i32, i32, i32, vp, vp, vp, i64, vp]
    lib.oracle_p_spmm.argtypes = [i32, i64, i64, i32, i32, i32, vp, vp, vp, i64, i64, vp, vp]
    lib.oracle_p_refine.argtypes = [i32, i64, i64, i32, i32, i32, vp, i64, vp, vp, vp]
    lib.oracle_spmm.argtypes = [i32, i64, i64, i32, i32, i32, vp, vp, vp, i64, i64,
                                vp, vp, i32]
    lib.oracle_spmm_points.argtypes = [i32, i64, i64, i32, i32, i32, vp, vp, vp, i64,
                                       i64, i64, vp, vp, vp, vp]
    for f in (lib.oracle_compress, lib.oracle_densify, lib.oracle_repack, lib.oracle_spmm,
              lib.oracle_spmm_points, lib.oracle_p_patterns, lib.oracle_p_compress,
              lib.oracle_p_densify, lib.oracle_p_spmm, lib.oracle_p_refine):
        f.restype = i32
    lib.oracle_half_to_float.argtypes = [ctypes.c_uint16]
    lib.oracle_half_to_float.restype = ctypes.c_float
    lib.oracle_double_to_half.argtypes = [ctypes.c_double]
    lib.oracle_double_to_half.restype = ctypes.c_uint16
    lib.oracle_float_to_half.argtypes = [ctypes.c_float]
    lib.oracle_float_to_half.restype = ctypes.c_uint16
    lib.oracle_round_to_half.argtypes = [vp, vp, i64]
    lib.oracle_gelu_f16.argtypes = [vp, vp, i64]
    lib.oracle_add_f16.argtypes = [vp, vp, vp, i64]
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.float16:
        return F16
    raise TypeError(f"oracle handles float32 and float16, got {a.dtype}")


def n_chunks(K: int, m: int) -> int:
    return -(-K // m)


def compress(W: np.ndarray, n: int, m: int, g: int):
    """Section 5.2 converter under the group reading: returns (values, indices).

    values  : M x (C*n), W's dtype; indices: (M/g) x (C*n) uint8 offsets.
    """
    W = np.ascontiguousarray(W)
    dt = _dtype_code(W)
    M, K = W.shape
    C = n_chunks(K, m)
    values = np.empty((M, C * n), dtype=W.dtype)
    indices = np.empty((max(M // g, 0), C * n), dtype=np.uint8)
    st = _load().oracle_compress(dt, M, K, n, m, g, _ptr(W), K, _ptr(values),
                                 _ptr(indices))
    if st:
        raise OracleError(st, "compress")
    return values, indices


def repack(W: np.ndarray, indices: np.ndarray, n: int, m: int, g: int) -> np.ndarray:
    """Fixed-mask repack (Section 5.3, a sparsifier keeping the existing
    format): W's entries at the positions `indices` selects, as values."""
    W = np.ascontiguousarray(W)
    indices = np.ascontiguousarray(indices, dtype=np.uint8)
    dt = _dtype_code(W)
    M, K = W.shape
    values = np.empty((M, n_chunks(K, m) * n), dtype=W.dtype)
    st = _load().oracle_repack(dt, M, K, n, m, g, _ptr(W), K, _ptr(indices), _ptr(values))
    if st:
        raise OracleError(st, "repack")
    return values


def densify(values: np.ndarray, indices: np.ndarray, K: int, n: int, m: int, g: int):
    """Section 5.2 conversion back to dense: returns (W_dense, mask)."""
    values = np.ascontiguousarray(values)
    indices = np.ascontiguousarray(indices, dtype=np.uint8)
    dt = _dtype_code(values)
    M = values.shape[0]
    out = np.empty((M, K), dtype=values.dtype)
    mask = np.empty((M, K), dtype=np.uint8)
    st = _load().oracle_densify(dt, M, K, n, m, g, _ptr(values), _ptr(indices),
                                _ptr(out), K, _ptr(mask))
    if st:
        raise OracleError(st, "densify")
    return out, mask.astype(bool)


def spmm(values, indices, X, K: int, n: int, m: int, g: int, nthreads: int = 0):
    """Y = densify(values, indices) @ X in binary64; returns (Y, B) with
    B = |W_s| @ |X| (the scale of the admissible rounding error)."""
    values = np.ascontiguousarray(values)
    indices = np.ascontiguousarray(indices, dtype=np.uint8)
    X = np.ascontiguousarray(X)
    if X.dtype != values.dtype:
        raise TypeError("values and X must share a dtype")
    dt = _dtype_code(values)
    M = values.shape[0]
    if X.shape[0] != K:
        raise ValueError("X must have K rows")
    N = X.shape[1]
    Y = np.empty((M, N), dtype=np.float64)
    B = np.empty((M, N), dtype=np.float64)
    st = _load().oracle_spmm(dt, M, K, n, m, g, _ptr(values), _ptr(indices), _ptr(X),
                             N, N, _ptr(Y), _ptr(B), nthreads)
    if st:
        raise OracleError(st, "spmm")
    return Y, B


def spmm_points(values, indices, X, K: int, n: int, m: int, g: int, rows, cols):
    """The oracle product at sampled outputs (rows[i], cols[i]); returns (Y, B)."""
    values = np.ascontiguousarray(values)
    indices = np.ascontiguousarray(indices, dtype=np.uint8)
    X = np.ascontiguousarray(X)
    if X.dtype != values.dtype:
        raise TypeError("values and X must share a dtype")
    dt = _dtype_code(values)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    M, N = values.shape[0], X.shape[1]
    Y = np.empty(rows.shape[0], dtype=np.float64)
    B = np.empty(rows.shape[0], dtype=np.float64)
    st = _load().oracle_spmm_points(dt, M, K, n, m, g, _ptr(values), _ptr(indices),
                                    _ptr(X), N, N, rows.shape[0], _ptr(rows),
                                    _ptr(cols), _ptr(Y), _ptr(B))
    if st:
        raise OracleError(st, "spmm_points")
    return Y, B


def half_to_float(bits: int) -> float:
    return float(_load().oracle_half_to_float(bits))


def double_to_half(x: float) -> int:
    return int(_load().oracle_double_to_half(x))


def float_to_half(x: float) -> int:
    return int(_load().oracle_float_to_half(x))


def round_to_half(x: np.ndarray) -> np.ndarray:
    """binary64 -> binary16, round to nearest even, elementwise."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().oracle_round_to_half(_ptr(x), _ptr(out), x.size)
    return out.view(np.float16)


def gelu_f16(x: np.ndarray) -> np.ndarray:
    """erf-form GELU in binary64, rounded once to binary16."""
    x = np.ascontiguousarray(x, dtype=np.float16)
    out = np.empty_like(x)
    _load().oracle_gelu_f16(_ptr(x), _ptr(out), x.size)
    return out


def add_f16(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """a + b, exact in binary64, rounded once to binary16."""
    a = np.ascontiguousarray(a, dtype=np.float16)
    b = np.ascontiguousarray(b, dtype=np.float16)
    out = np.empty_like(a)
    _load().oracle_add_f16(_ptr(a), _ptr(b), _ptr(out), a.size)
    return out


def energy(W: np.ndarray, values: np.ndarray) -> float:
    """Section 6.1 energy: L1 of the pruned tensor over L1 of the original."""
    return float(np.abs(values.astype(np.float64)).sum() /
                 np.abs(W.astype(np.float64)).sum())


def linear_stack_layer(x: np.ndarray, packed: dict, n: int, m: int, g: int):
    """One layer of the BERT-base encoder linear stack in binary16 storage.

    x: 768 x T binary16 activations (features x tokens).  ``packed`` maps
    'qkv', 'ao', 'up', 'down' to (values, indices, K).  Attention itself is
    omitted: the attention-output projection reads the V third of the QKV
    output.  Residual sums follow BERT's encoder block:
        h = x + AO(V(x)),   x' = h + Down(GELU(Up(h))).
    Every product is the binary64 oracle product rounded once to binary16.
    """
    def lin(name, inp):
        v, idx, K = packed[name]
        Y, _ = spmm(v, idx, inp, K, n, m, g)
        return round_to_half(Y)

    qkv = lin("qkv", x)
    d = x.shape[0]
    vpart = np.ascontiguousarray(qkv[2 * d:3 * d])
    h = add_f16(x, lin("ao", vpart))
    u = gelu_f16(lin("up", h))
    return add_f16(h, lin("down", u))


# ------------------------------------------------ the paper's chunked layout

def p_patterns(m: int, n: int) -> np.ndarray:
    """The C(m, n) patterns in revolving-door order (P x n offsets)."""
    P = math.comb(m, n)
    out = np.zeros((max(P, 1), n), dtype=np.uint8)
    st = _load().oracle_p_patterns(m, n, _ptr(out))
    if st:
        raise OracleError(st, "p_patterns")
    return out


def p_compress(W: np.ndarray, n: int, m: int, g: int):
    """Section 5.2 CPU converter into the chunked layout: (values, index).

    values: M x (K/m * n), rows of each chunk in pattern order; index: M x (K/m)
    uint8, the chunk row of the block at each position."""
    W = np.ascontiguousarray(W)
    dt = _dtype_code(W)
    M, K = W.shape
    B = K // m if m else 0
    values = np.empty((M, B * n), dtype=W.dtype)
    index = np.empty((M, B), dtype=np.uint8)
    st = _load().oracle_p_compress(dt, M, K, n, m, g, _ptr(W), K, _ptr(values), _ptr(index))
    if st:
        raise OracleError(st, "p_compress")
    return values, index


def p_densify(values: np.ndarray, index: np.ndarray, K: int, n: int, m: int, g: int):
    values = np.ascontiguousarray(values)
    index = np.ascontiguousarray(index, dtype=np.uint8)
    dt = _dtype_code(values)
    M = values.shape[0]
    out = np.empty((M, K), dtype=values.dtype)
    mask = np.empty((M, K), dtype=np.uint8)
    st = _load().oracle_p_densify(dt, M, K, n, m, g, _ptr(values), _ptr(index), _ptr(out), K,
                                  _ptr(mask))
    if st:
        raise OracleError(st, "p_densify")
    return out, mask.astype(bool)


def p_spmm(values, index, X, K: int, n: int, m: int, g: int):
    """Y = W_s X (binary64) for the chunked layout, and B = |W_s| |X|."""
    values = np.ascontiguousarray(values)
    index = np.ascontiguousarray(index, dtype=np.uint8)
    X = np.ascontiguousarray(X)
    dt = _dtype_code(values)
    M, N = values.shape[0], X.shape[1]
    Y = np.empty((M, N), dtype=np.float64)
    Bnd = np.empty((M, N), dtype=np.float64)
    st = _load().oracle_p_spmm(dt, M, K, n, m, g, _ptr(values), _ptr(index), _ptr(X), N, N,
                               _ptr(Y), _ptr(Bnd))
    if st:
        raise OracleError(st, "p_spmm")
    return Y, Bnd


def p_refine(W: np.ndarray, index: np.ndarray, n: int, m: int, g: int):
    """The swap search of Section 5.2 from the packing `index` (this module's
    fixed-order reading): returns (values, index, rounds of the slowest chunk)."""
    W = np.ascontiguousarray(W)
    dt = _dtype_code(W)
    M, K = W.shape
    idx = np.array(index, dtype=np.uint8, copy=True, order="C")
    values = np.empty((M, (K // m) * n), dtype=W.dtype)
    rounds = ctypes.c_int(0)
    st = _load().oracle_p_refine(dt, M, K, n, m, g, _ptr(W), K, _ptr(values), _ptr(idx),
                                 ctypes.byref(rounds))
    if st:
        raise OracleError(st, "p_refine")
    return values, idx, rounds.value
