"""ctypes loader for libmosaic.so (the C ABI of include/mosaic.h).

The library must have been built in-tree (``python -m
paper_2607_29221_amd.build``); there is no fallback implementation, so a
missing library is an error.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmosaic.so")
_DEFAULT_LIB_PATH = LIB_PATH

c_i32 = ctypes.c_int32
c_i64 = ctypes.c_int64
c_u32 = ctypes.c_uint32
c_u64 = ctypes.c_uint64
c_ptr = ctypes.c_void_p


class MosaicRng(ctypes.Structure):
    _fields_ = [
        ("seed", c_u64),
        ("stream", c_u32),
        ("instance", c_u32),
        ("dist", c_i32),
        ("bound", c_i32),
        ("sigma", ctypes.c_double),
        ("log2_inv_density", c_i32),
        ("transposed", c_i32),
        ("row_weight", c_i32),
    ]


# name -> argument types (all return mosaic_status as int32 unless listed)
_SIGNATURES = {
    "mosaic_abi_version": ([], c_i32),
    "mosaic_last_error_message": ([], ctypes.c_char_p),
    "mosaic_last_error_string": ([], ctypes.c_char_p),
    "mosaic_dgauss_thresholds": ([ctypes.c_double, c_i32, ctypes.POINTER(c_u64)], c_i32),
    "mosaic_sample": ([ctypes.POINTER(MosaicRng), c_i64, c_i64, c_ptr, c_i64, c_ptr, c_i64, c_ptr], c_i32),
    "mosaic_mask": ([c_ptr, c_i32, c_i64, c_i64, c_ptr, c_i64, ctypes.POINTER(MosaicRng), c_i64, c_i64,
                     c_ptr, c_i64, c_ptr, c_i64, c_ptr], c_i32),
    "mosaic_masked_matmul": ([c_ptr, c_i64, c_ptr, c_i64, c_i64, c_i64, c_i64, c_ptr, c_i64, c_ptr], c_i32),
    "mosaic_masked_matmul_words": ([c_ptr, c_i64, c_ptr, c_i64, c_i64, c_i64, c_i64, c_ptr, c_i64, c_i32, c_ptr],
                                   c_i32),
    "mosaic_integrity_check": ([c_ptr, c_i64, c_ptr, c_i64, c_ptr, c_i64, c_ptr, c_i64, c_i64, c_i64, c_i64,
                                c_i64, c_ptr, c_i64, c_ptr, c_ptr], c_i32),
    "mosaic_unmask": ([c_ptr, c_i64, c_ptr, c_i64, c_ptr, c_i64, c_ptr, c_i64, c_i64, c_i64, c_i64,
                       c_ptr, c_i64, c_ptr, c_ptr, c_ptr, c_ptr, c_i64, c_ptr], c_i32),
    "mosaic_unmask_words": ([c_ptr, c_i64, c_ptr, c_i64, c_ptr, c_i64, c_ptr, c_i64, c_i64, c_i64, c_i64,
                             c_ptr, c_i64, c_ptr, c_ptr, c_ptr, c_ptr, c_i64, c_ptr], c_i32),
    "mosaic_sample_signs": ([ctypes.POINTER(MosaicRng), c_i64, c_ptr, c_ptr], c_i32),
    "mosaic_rotate_quantize_mask": ([c_ptr, c_i64, c_i64, c_i64, c_i64, c_ptr, c_i32, c_ptr, c_i64,
                                     ctypes.POINTER(MosaicRng), c_ptr, c_i64, c_ptr, c_ptr], c_i32),
    "mosaic_count_mismatches": ([c_ptr, c_i64, c_ptr, c_i64, c_i64, c_i64, c_ptr, c_ptr], c_i32),
    "mosaic_sparse_csr_count": ([ctypes.POINTER(MosaicRng), c_i64, c_i64, c_ptr, c_ptr], c_i32),
    "mosaic_sparse_csr_fill": ([ctypes.POINTER(MosaicRng), c_i64, c_i64, c_ptr, c_ptr, c_ptr, c_ptr], c_i32),
    "mosaic_sparse_gather_rows": ([c_i64, c_ptr, c_ptr, c_ptr, c_ptr, c_i64, c_i64, c_ptr, c_i64, c_i32, c_ptr],
                                  c_i32),
    "mosaic_sparse_stream_gather_rows": ([ctypes.POINTER(MosaicRng), c_i64, c_i64, c_ptr, c_i64, c_i64, c_ptr, c_i64,
                                          c_i32, c_ptr], c_i32),
    "mosaic_sparse_gather_cols": ([c_i64, c_i64, c_ptr, c_ptr, c_ptr, c_ptr, c_i64, c_ptr, c_i64, c_i32,
                                   c_ptr, c_ptr, c_ptr, c_ptr, c_i64, c_ptr], c_i32),
    "mosaic_hadamard_rotate": ([c_ptr, c_i64, c_ptr, c_i64, c_i64, c_i64, c_i64, c_ptr, c_i32, c_ptr], c_i32),
    "mosaic_hadamard28_rotate": ([c_ptr, c_i64, c_ptr, c_i64, c_i64, c_i64, c_ptr, c_i32, c_ptr], c_i32),
    "mosaic_probe_mfma_i8": ([c_i32, c_i64, c_ptr, ctypes.POINTER(c_i64), c_ptr], c_i32),
    "mosaic_quantize_rows": ([c_ptr, c_i64, c_i64, c_i64, c_i32, c_ptr, c_i64, c_ptr, c_i64, c_ptr, c_ptr],
                             c_i32),
}

EXPORTED = tuple(_SIGNATURES)

_lib = None


def stale_reason() -> Optional[str]:
    """Why the in-tree library does not match the sources, or None. The build
    writes a digest of its sources beside the library; a library built from
    other sources (an edit after the last build) would run other kernels
    than the ones in the tree."""
    from . import build as _build
    if not os.path.exists(_build.STAMP):
        return f"{_build.STAMP} is missing"
    with open(_build.STAMP) as f:
        stamp = f.read().strip()
    if stamp != _build.source_digest():
        return "the sources under csrc/ or include/ changed after the last build"
    return None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2607_29221_amd.build`")
        if LIB_PATH == _DEFAULT_LIB_PATH:
            why = stale_reason()
            if why is not None:
                raise RuntimeError(f"{LIB_PATH} is stale ({why}): run `python -m paper_2607_29221_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        _lib = lib
    return _lib
