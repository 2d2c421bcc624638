"""Oracle for the W4A4 sparse product and its epilogue (TEST INFRASTRUCTURE ONLY).

The SpMM result has a plain definition because IE-BME is lossless: Y = W X
over the decoded INT4 weights (Section VI, kernel algorithm: the kernel's
output matrix Y). Here that definition is written out twice: in plain C with
int64 accumulation (``matmul_i64.c``, used for large cases and for the CPU
baseline) and as numpy int64 matmul. The optional dequantisation epilogue is
not in the paper; it is read as one float32 multiply per output,
fl32(fl32(Y[m, n]) * scale[m]), rounded to nearest even.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this package.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "matmul_i64.c")
_LIB = os.path.join(_HERE, "_liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (plain -O2, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        lib.oracle_matmul_i64.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p]
        lib.oracle_matmul_i64.restype = None
        lib.oracle_max_threads.restype = ctypes.c_int
        lib.oracle_set_threads.argtypes = [ctypes.c_int]
        lib.oracle_set_threads.restype = None
        _lib = lib
    return _lib


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def set_threads(n: int) -> None:
    """Threads the C product uses from now on (for timing it on one core)."""
    _load().oracle_set_threads(int(n))


def matmul_c(W: np.ndarray, Xt: np.ndarray) -> np.ndarray:
    """Y[m, n] = sum_k W[m, k] * Xt[n, k] in int64, by the plain C loop."""
    W = np.ascontiguousarray(W, dtype=np.int8)
    Xt = np.ascontiguousarray(Xt, dtype=np.int8)
    M, K = W.shape
    N, K2 = Xt.shape
    if K != K2:
        raise ValueError("inner dimensions differ")
    Y = np.empty((M, N), dtype=np.int64)
    _load().oracle_matmul_i64(W.ctypes.data, Xt.ctypes.data, M, K, N, Y.ctypes.data)
    return Y


def matmul_np(W: np.ndarray, Xt: np.ndarray) -> np.ndarray:
    """The same product with numpy's int64 matmul."""
    return np.asarray(W, dtype=np.int64) @ np.asarray(Xt, dtype=np.int64).T


def to_int32(Y: np.ndarray) -> np.ndarray:
    """The kernel's INT32 result; the int64 sum must fit."""
    if Y.size and (Y.min() < np.iinfo(np.int32).min or Y.max() > np.iinfo(np.int32).max):
        raise OverflowError("product does not fit in int32")
    return Y.astype(np.int32)


def dequant(Y: np.ndarray, scale: np.ndarray) -> np.ndarray:
    """fl32(fl32(Y[m, n]) * scale[m]) for Y of shape (M, N)."""
    Yf = np.asarray(Y).astype(np.float32)     # exact: |Y| < 2**24
    return Yf * np.asarray(scale, dtype=np.float32)[:, None]
