"""Loader of the oracle's C stream generator (oracle/c/philox_stream.c),
compiled with gcc into oracle/c/libphilox_stream.so on first use."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c")
_SRC = os.path.join(_DIR, "philox_stream.c")
_LIB = os.path.join(_DIR, "libphilox_stream.so")
_lib = None


def build() -> str:
    tmp = _LIB + f".tmp{os.getpid()}"
    subprocess.run(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", tmp, _SRC], check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB)
        lib.oracle_stream_words.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64,
                                            ctypes.c_uint64, ctypes.c_void_p]
        lib.oracle_stream_words.restype = None
        _lib = lib
    return _lib


def stream_words(seed: int, stream: int, instance: int, t0: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.uint32)
    _load().oracle_stream_words(seed & 0xFFFFFFFFFFFFFFFF, stream, instance, t0, count, out.ctypes.data)
    return out
