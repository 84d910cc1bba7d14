"""Loader of the oracle's plain C leg (oracle/c/ring_oracle.c: ring products
over Z_{2^32} and the float64 rotation, OpenMP over rows), compiled with gcc
into oracle/c/libring_oracle.so on first use. Test infrastructure and the
CPU baseline only."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c")
_SRC = os.path.join(_DIR, "ring_oracle.c")
_LIB = os.path.join(_DIR, "libring_oracle.so")
_lib = None


def build() -> str:
    tmp = _LIB + f".tmp{os.getpid()}"
    subprocess.run(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"], check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB)
        i64, p = ctypes.c_int64, ctypes.c_void_p
        lib.oracle_ring_matmul_nt.argtypes = [p, i64, p, i64, p, i64, i64, i64, i64]
        lib.oracle_ring_matmul_nt.restype = None
        lib.oracle_rotate_rows.argtypes = [p, i64, i64, p, ctypes.c_int]
        lib.oracle_rotate_rows.restype = None
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def threads() -> int:
    return int(_load().oracle_threads())


def ring_matmul_nt(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """a @ b.T over Z_{2^32}; a (m x k), b (n x k) uint32."""
    a = np.ascontiguousarray(a, dtype=np.uint32)
    b = np.ascontiguousarray(b, dtype=np.uint32)
    m, k = a.shape
    n, k2 = b.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    c = np.empty((m, n), dtype=np.uint32)
    _load().oracle_ring_matmul_nt(a.ctypes.data, k, b.ctypes.data, k, c.ctypes.data, n, m, n, k)
    return c


def rotate_rows(x: np.ndarray, signs=None, inverse: bool = False) -> np.ndarray:
    """Row-wise random Hadamard rotation (forward or inverse) in float64."""
    y = np.array(x, dtype=np.float64, order="C", copy=True)
    rows, n = y.shape
    if n & (n - 1):
        raise ValueError("length must be a power of two")
    s = None if signs is None else np.ascontiguousarray(signs, dtype=np.int8)
    _load().oracle_rotate_rows(y.ctypes.data, rows, n, None if s is None else s.ctypes.data, 1 if inverse else 0)
    return y
