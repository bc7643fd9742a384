"""Python entry points of the GEMM oracle (oracle/gemm_ref.c via ctypes).

TEST INFRASTRUCTURE ONLY -- never called by the product.

``gemm_ref_rows`` and ``gemm_ref_points`` return the fp64 product C = A * B of
the bf16 inputs (Section II.A; overwrite semantics of Listing 1) and the scale
R = |A| * |B| for the same elements.  ``build`` compiles the C file with gcc.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gemm_ref.c")
_LIB = os.path.join(_HERE, "_gemm_ref.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile oracle/gemm_ref.c into oracle/_gemm_ref.so with gcc + OpenMP."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
                        "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build(force=False)
            lib = ctypes.CDLL(_LIB)
            i64, p = ctypes.c_int64, ctypes.c_void_p
            lib.gemm_ref_rows.argtypes = [i64, i64, i64, i64, p, i64, p, i64, p, p]
            lib.gemm_ref_rows.restype = None
            lib.gemm_ref_points.argtypes = [i64, p, p, i64, p, i64, p, i64, p, p]
            lib.gemm_ref_points.restype = None
            lib.gemm_ref_threads.argtypes = []
            lib.gemm_ref_threads.restype = ctypes.c_int
            _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _check_operands(A, B, K, lda, ldb, rows_needed, cols_needed):
    A = np.ascontiguousarray(A, dtype=np.uint16).reshape(-1)
    B = np.ascontiguousarray(B, dtype=np.uint16).reshape(-1)
    if K > 0:
        if rows_needed > 0 and A.size < (rows_needed - 1) * lda + K:
            raise ValueError("A is too small for the requested rows")
        if cols_needed > 0 and B.size < (K - 1) * ldb + cols_needed:
            raise ValueError("B is too small for the requested columns")
    return A, B


def gemm_ref_rows(A, B, N: int, K: int, lda: int, ldb: int, row0: int = 0, nrows: int = None,
                  M: int = None):
    """Rows [row0, row0+nrows) of C = A*B and R = |A|*|B| as fp64 (nrows x N)."""
    if nrows is None:
        nrows = M - row0
    A, B = _check_operands(A, B, K, lda, ldb, row0 + nrows, N)
    C = np.empty((nrows, N), dtype=np.float64)
    R = np.empty((nrows, N), dtype=np.float64)
    if nrows > 0 and N > 0:
        _load().gemm_ref_rows(row0, nrows, N, K, _ptr(A), lda, _ptr(B), ldb, _ptr(C), _ptr(R))
    return C, R


def gemm_ref_points(A, B, K: int, lda: int, ldb: int, rows, cols):
    """C[rows[p], cols[p]] and R[rows[p], cols[p]] as fp64 vectors."""
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    if rows.shape != cols.shape:
        raise ValueError("rows and cols differ in shape")
    A, B = _check_operands(A, B, K, lda, ldb, int(rows.max()) + 1 if rows.size else 0,
                           int(cols.max()) + 1 if cols.size else 0)
    C = np.empty(rows.shape, dtype=np.float64)
    R = np.empty(rows.shape, dtype=np.float64)
    if rows.size:
        _load().gemm_ref_points(rows.size, _ptr(rows), _ptr(cols), K, _ptr(A), lda, _ptr(B), ldb,
                                _ptr(C), _ptr(R))
    return C, R


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().gemm_ref_threads())
