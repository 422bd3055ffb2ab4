"""Loader for the oracle's plain C products (oracle/linear.c).

TEST INFRASTRUCTURE.  Builds the library with gcc on first use if it is
missing or older than its source; falls back to NumPy if no compiler works.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "linear.c")
_LIB = os.path.join(_HERE, "liboracle_linear.so")
_lib = None
_tried = False


def build(force: bool = False) -> str:
    """Compile linear.c → liboracle_linear.so (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib, _tried
    if _lib is None and not _tried:
        _tried = True
        try:
            path = build()
            L = ctypes.CDLL(path)
            for name in ("oracle_linear_bf16", "oracle_linear_f32"):
                fn = getattr(L, name)
                fn.restype = None
                fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                               ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]
            _lib = L
        except Exception:  # no compiler: NumPy path below
            _lib = None
    return _lib


def linear(W: np.ndarray, X: np.ndarray, use_c: bool = True) -> np.ndarray:
    """Y = X @ W^T in fp64.  W: [N, K] stored bf16 bits (uint16) or fp32/fp64."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    M, K = X.shape
    N = W.shape[0]
    assert W.shape[1] == K, (W.shape, X.shape)
    L = lib() if use_c else None
    if L is not None and W.dtype in (np.uint16, np.float32):
        W = np.ascontiguousarray(W)
        Y = np.empty((M, N), dtype=np.float64)
        fn = L.oracle_linear_bf16 if W.dtype == np.uint16 else L.oracle_linear_f32
        fn(W.ctypes.data, X.ctypes.data, Y.ctypes.data, M, N, K)
        return Y
    # NumPy: widen W to fp64 in row chunks and multiply
    Y = np.empty((M, N), dtype=np.float64)
    step = max(1, (1 << 24) // max(K, 1))
    for n0 in range(0, N, step):
        Wc = widen(W[n0:n0 + step])
        Y[:, n0:n0 + step] = X @ Wc.T
    return Y


def widen(a: np.ndarray) -> np.ndarray:
    """Exact fp64 value of stored data (bf16 bit patterns or floats)."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)
