"""Python binding of the MOSAIC C ABI (include/mosaic.h).

Each function has the name of the ABI entry point it calls and only marshals
arguments: torch tensors (device memory, on the current HIP stream) become
pointers, leading dimensions and sizes. All arithmetic runs in the HIP
kernels of libmosaic.so.

Digit-layout matrices are ``Digits`` views: an int8 tensor of shape
(rows, pitch) plus a column offset (a multiple of 64), so several factors can
share one buffer side by side.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import List, Optional, Sequence

import torch

from . import _lib

DIST_ZERO, DIST_UNIFORM, DIST_DGAUSS, DIST_SPARSE, DIST_WEIGHT = 0, 1, 2, 3, 4
DT_I8, DT_I16, DT_I32, DT_U32 = 0, 1, 2, 3
STATUS_OK, STATUS_INVALID_ARG, STATUS_UNSUPPORTED, STATUS_HIP = 0, -1, -2, -3
_TORCH_DT = {torch.int8: DT_I8, torch.int16: DT_I16, torch.int32: DT_I32}


class MosaicError(RuntimeError):
    def __init__(self, status: int, name: str):
        msg = _lib.load().mosaic_last_error_message().decode(errors="replace")
        super().__init__(f"{name} failed with status {status}: {msg}")
        self.status = status


def _check(status: int, name: str) -> None:
    if status != 0:
        raise MosaicError(status, name)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def padded_k(k: int) -> int:
    return 64 * ((k + 63) // 64)


# Host-side shape checks before any launch: the C ABI sees only pointers and
# sizes, so a tensor smaller than the sizes passed would be read or written
# past its end on the GPU. These raise ValueError instead.
def _need(t: Optional[torch.Tensor], rows: int, cols: int, name: str, dtypes=None, optional: bool = True) -> None:
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if dtypes is not None and t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if rows == 0 or cols == 0:
        return
    if t.dim() == 1:
        if rows * cols > t.numel() or (rows > 1 and cols > 1):
            raise ValueError(f"{name} holds {t.numel()} elements, needs {rows} x {cols}")
        return
    if t.dim() != 2:
        raise ValueError(f"{name} must be a matrix")
    if t.shape[0] < rows or t.shape[1] < cols:
        raise ValueError(f"{name} is {tuple(t.shape)}, needs at least ({rows}, {cols})")
    if cols > 1 and t.stride(1) != 1:
        raise ValueError(f"{name} must have contiguous rows")


def _need_dig(d: Optional["Digits"], rows: int, cols: int, name: str, optional: bool = True) -> None:
    if d is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not d.buf.is_cuda or d.buf.dtype != torch.int8 or d.buf.dim() != 2 or d.buf.stride(1) != 1:
        raise ValueError(f"{name} must be a row-contiguous int8 device matrix")
    if rows == 0 or cols == 0:
        return
    if d.rows < rows or d.col0 % 64 or 4 * (d.col0 + padded_k(cols)) > d.pitch:
        raise ValueError(f"{name} ({d.rows} rows, pitch {d.pitch}, column {d.col0}) cannot hold {rows} x {cols} digits")


_INT = (torch.int32,)


@dataclass
class Digits:
    """rows x cols ring matrix in digit layout, at column ``col0`` of ``buf``."""
    buf: torch.Tensor          # int8, (rows, pitch)
    cols: int
    col0: int = 0

    @property
    def rows(self) -> int:
        return self.buf.shape[0]

    @property
    def pitch(self) -> int:
        return self.buf.shape[1]

    @property
    def ptr(self) -> int:
        return self.buf.data_ptr() + 4 * self.col0

    @staticmethod
    def empty(rows: int, cols: int, device="cuda") -> "Digits":
        return Digits(torch.empty((rows, 4 * padded_k(cols)), dtype=torch.int8, device=device), cols)

    @staticmethod
    def concat(rows: int, cols: Sequence[int], device="cuda") -> List["Digits"]:
        """Factors side by side in one buffer (each padded to 64 columns)."""
        total = sum(padded_k(c) for c in cols)
        buf = torch.empty((rows, 4 * max(total, 64)), dtype=torch.int8, device=device)
        out, off = [], 0
        for c in cols:
            out.append(Digits(buf, c, off))
            off += padded_k(c)
        return out

    def whole(self, cols: int) -> "Digits":
        """The full buffer seen as one matrix of ``cols`` columns from column 0."""
        return Digits(self.buf, cols, 0)


def rng(seed: int, stream: int, instance: int, dist: int, sigma: float = 0.5, bound: int = 4,
        log2_inv_density: int = 6, transposed: bool = False, row_weight: int = 0) -> _lib.MosaicRng:
    return _lib.MosaicRng(seed=seed & 0xFFFFFFFFFFFFFFFF, stream=stream, instance=instance, dist=dist,
                          bound=bound, sigma=sigma, log2_inv_density=log2_inv_density,
                          transposed=1 if transposed else 0, row_weight=row_weight)


def mosaic_abi_version() -> int:
    return _lib.load().mosaic_abi_version()


def mosaic_dgauss_thresholds(sigma: float, bound: int) -> List[int]:
    arr = (ctypes.c_uint64 * max(2 * bound, 1))()
    _check(_lib.load().mosaic_dgauss_thresholds(sigma, bound, arr), "mosaic_dgauss_thresholds")
    return [int(arr[i]) for i in range(2 * bound)]


def mosaic_sample(r: _lib.MosaicRng, rows: int, cols: int, out: Optional[torch.Tensor] = None,
                  out_dig: Optional[Digits] = None) -> None:
    _need(out, rows, cols, "out", _INT)
    _need_dig(out_dig, rows, cols, "out_dig")
    ldo = out.stride(0) if out is not None else 0
    _check(_lib.load().mosaic_sample(ctypes.byref(r), rows, cols, _ptr(out), ldo,
                                     out_dig.ptr if out_dig else None, out_dig.pitch if out_dig else 0,
                                     _stream()), "mosaic_sample")


def mosaic_mask(x: Optional[torch.Tensor], u: Optional[torch.Tensor], noise: Optional[_lib.MosaicRng],
                rows: int, cols: int, out: Optional[torch.Tensor] = None,
                out_dig: Optional[Digits] = None, x_transposed: bool = False) -> None:
    """out = x + u + noise (mod 2^32). ``x_transposed`` reads x[j, i] for
    element (i, j) (x then has shape (cols, rows))."""
    if x is not None:
        if x.dtype not in _TORCH_DT or not x.is_cuda or x.dim() != 2:
            raise ValueError("x must be an int8/int16/int32 device matrix")
        xr, xc = (cols, rows) if x_transposed else (rows, cols)
        if x.shape[0] < xr or x.shape[1] < xc:
            raise ValueError(f"x is {tuple(x.shape)}, needs at least ({xr}, {xc})")
        dt = _TORCH_DT[x.dtype]   # int32 and uint32 embed identically into the ring
        rs, cs = (x.stride(1), x.stride(0)) if x_transposed else (x.stride(0), x.stride(1))
    else:
        dt, rs, cs = DT_U32, 0, 0
    _need(u, rows, cols, "u", _INT)
    _need(out, rows, cols, "out", _INT)
    _need_dig(out_dig, rows, cols, "out_dig")
    ldu = u.stride(0) if u is not None else 0
    ldo = out.stride(0) if out is not None else 0
    _check(_lib.load().mosaic_mask(_ptr(x), dt, rs, cs, _ptr(u), ldu,
                                   ctypes.byref(noise) if noise is not None else None, rows, cols,
                                   _ptr(out), ldo, out_dig.ptr if out_dig else None,
                                   out_dig.pitch if out_dig else 0, _stream()), "mosaic_mask")


def mosaic_masked_matmul(a: Digits, b: Digits, M: int, N: int, K: int, c: torch.Tensor) -> None:
    """c[:M, :N] = A B^T over Z_{2^32} (c is an int32 tensor holding ring words)."""
    _need_dig(a, M, K, "a", optional=False)
    _need_dig(b, N, K, "b", optional=False)
    _need(c, M, N, "c", _INT, optional=False)
    _check(_lib.load().mosaic_masked_matmul(a.ptr, a.pitch, b.ptr, b.pitch, M, N, K, c.data_ptr(),
                                            c.stride(0), _stream()), "mosaic_masked_matmul")


def mosaic_masked_matmul_words(a: Digits, b: torch.Tensor, M: int, N: int, K: int, c: torch.Tensor,
                               accumulate: bool = False) -> None:
    """c[:M, :N] (+)= A B^T over Z_{2^32} with B (N x K) given as ring words
    (an int32 tensor); A has at most 64 rows."""
    _need_dig(a, M, K, "a", optional=False)
    _need(b, N, K, "b", _INT, optional=False)
    _need(c, M, N, "c", _INT, optional=False)
    _check(_lib.load().mosaic_masked_matmul_words(a.ptr, a.pitch, b.data_ptr(), b.stride(0), M, N, K, c.data_ptr(),
                                                  c.stride(0), 1 if accumulate else 0, _stream()),
           "mosaic_masked_matmul_words")


def mosaic_integrity_check(ct: Digits, a: Digits, v: Digits, yq: torch.Tensor, t: int, M: int, K: int, NR: int,
                           d: torch.Tensor, count: torch.Tensor) -> None:
    """d = c^T A'^T - V [Y' | Q]^T (t x M) and count[0] = its nonzero entries,
    with [Y' | Q] given as the ring words of yq's first NR columns."""
    _need_dig(ct, t, K, "ct", optional=False)
    _need_dig(a, M, K, "a", optional=False)
    _need_dig(v, t, NR, "v", optional=False)
    _need(yq, M, NR, "yq", _INT, optional=False)
    _need(d, t, M, "d", _INT, optional=False)
    if count.dtype != torch.int64 or count.numel() < 1 or not count.is_cuda:
        raise ValueError("count must be an int64 device tensor")
    _check(_lib.load().mosaic_integrity_check(ct.ptr, ct.pitch, a.ptr, a.pitch, v.ptr, v.pitch, yq.data_ptr(),
                                              yq.stride(0), t, M, K, NR, d.data_ptr(), d.stride(0),
                                              count.data_ptr(), _stream()), "mosaic_integrity_check")


def mosaic_unmask(ym: torch.Tensor, kc: Optional[torch.Tensor], q: Optional[Digits], l: Optional[Digits],
                  M: int, N: int, R: int, y: Optional[torch.Tensor] = None,
                  s_rows: Optional[torch.Tensor] = None, s_cols: Optional[torch.Tensor] = None,
                  y_f32: Optional[torch.Tensor] = None, bias: Optional[torch.Tensor] = None) -> None:
    _need(ym, M, N, "ym", _INT, optional=False)
    _need(kc, M, N, "kc", _INT)
    if R > 0:
        _need_dig(q, M, R, "q", optional=False)
        _need_dig(l, N, R, "l", optional=False)
    _need(y, M, N, "y", _INT)
    _need(y_f32, M, N, "y_f32", (torch.float32,))
    if y_f32 is not None:
        _need(s_rows, 1, M, "s_rows", (torch.float32,), optional=False)
        _need(s_cols, 1, N, "s_cols", (torch.float32,), optional=False)
    _need(bias, 1, N, "bias", (torch.float32,))
    _check(_lib.load().mosaic_unmask(ym.data_ptr(), ym.stride(0), _ptr(kc), kc.stride(0) if kc is not None else 0,
                                     q.ptr if q else None, q.pitch if q else 0,
                                     l.ptr if l else None, l.pitch if l else 0, M, N, R,
                                     _ptr(y), y.stride(0) if y is not None else 0,
                                     _ptr(s_rows), _ptr(s_cols), _ptr(bias), _ptr(y_f32),
                                     y_f32.stride(0) if y_f32 is not None else 0, _stream()), "mosaic_unmask")


def mosaic_unmask_words(ym: torch.Tensor, kc: Optional[torch.Tensor], q: Optional[torch.Tensor],
                        l: Optional[Digits], M: int, N: int, R: int, y: Optional[torch.Tensor] = None,
                        s_rows: Optional[torch.Tensor] = None, s_cols: Optional[torch.Tensor] = None,
                        y_f32: Optional[torch.Tensor] = None, bias: Optional[torch.Tensor] = None) -> None:
    """mosaic_unmask with q (M x R) as ring words, e.g. the Q columns of the
    server's [Y' | Q]; at most 16 rows."""
    _need(ym, M, N, "ym", _INT, optional=False)
    _need(kc, M, N, "kc", _INT)
    if R > 0:
        _need(q, M, R, "q", _INT, optional=False)
        _need_dig(l, N, R, "l", optional=False)
    _need(y, M, N, "y", _INT)
    _need(y_f32, M, N, "y_f32", (torch.float32,))
    if y_f32 is not None:
        _need(s_rows, 1, M, "s_rows", (torch.float32,), optional=False)
        _need(s_cols, 1, N, "s_cols", (torch.float32,), optional=False)
    _need(bias, 1, N, "bias", (torch.float32,))
    _check(_lib.load().mosaic_unmask_words(ym.data_ptr(), ym.stride(0), _ptr(kc),
                                           kc.stride(0) if kc is not None else 0,
                                           _ptr(q), q.stride(0) if q is not None else 0,
                                           l.ptr if l else None, l.pitch if l else 0, M, N, R,
                                           _ptr(y), y.stride(0) if y is not None else 0,
                                           _ptr(s_rows), _ptr(s_cols), _ptr(bias), _ptr(y_f32),
                                           y_f32.stride(0) if y_f32 is not None else 0, _stream()),
           "mosaic_unmask_words")


def mosaic_rotate_quantize_mask(x: torch.Tensor, qmax: int, out_dig: Digits, block: Optional[int] = None,
                                signs: Optional[torch.Tensor] = None, u: Optional[torch.Tensor] = None,
                                noise: Optional[_lib.MosaicRng] = None,
                                scale: Optional[torch.Tensor] = None) -> None:
    """Fused rotate + quantise + mask of Pi_Sec-Linear's input: digits of
    round(R x / s) + u + noise for every row of x, and the row scales."""
    rows, n = x.shape
    _need(x, rows, n, "x", (torch.float32,), optional=False)
    _need_dig(out_dig, rows, n, "out_dig", optional=False)
    _need(u, rows, n, "u", _INT)
    _need(scale, 1, rows, "scale", (torch.float32,))
    _need(signs, 1, n, "signs", (torch.int8,))
    _check(_lib.load().mosaic_rotate_quantize_mask(x.data_ptr(), x.stride(0), rows, n, n if block is None else block,
                                                   _ptr(signs), qmax, _ptr(u), u.stride(0) if u is not None else 0,
                                                   ctypes.byref(noise) if noise is not None else None,
                                                   out_dig.ptr, out_dig.pitch, _ptr(scale), _stream()),
           "mosaic_rotate_quantize_mask")


@dataclass
class SparseRows:
    """Compressed rows of a sparse ring matrix (rows x cols) on the device."""
    row_ptr: torch.Tensor      # int64, rows + 1
    col_idx: torch.Tensor      # int32, capacity >= nnz
    values: torch.Tensor       # int32 holding uint32 ring values
    rows: int
    cols: int


def mosaic_sparse_csr(r: _lib.MosaicRng, rows: int, cols: int, exact: bool = True, device="cuda") -> SparseRows:
    """Compressed rows of the SPARSE or WEIGHT stream matrix of ``r``. With
    ``exact`` the arrays are sized to the nonzero count (one device-to-host
    read for SPARSE; rows * t for WEIGHT); otherwise to the bound rows * cols
    (no synchronisation)."""
    row_ptr = torch.empty(rows + 1, dtype=torch.int64, device=device)
    _check(_lib.load().mosaic_sparse_csr_count(ctypes.byref(r), rows, cols, row_ptr.data_ptr(), _stream()),
           "mosaic_sparse_csr_count")
    if r.dist == DIST_WEIGHT:
        cap = rows * r.row_weight
    else:
        cap = int(row_ptr[rows].item()) if exact else rows * cols
    col_idx = torch.empty(max(cap, 1), dtype=torch.int32, device=device)
    values = torch.empty(max(cap, 1), dtype=torch.int32, device=device)
    _check(_lib.load().mosaic_sparse_csr_fill(ctypes.byref(r), rows, cols, row_ptr.data_ptr(), col_idx.data_ptr(),
                                              values.data_ptr(), _stream()), "mosaic_sparse_csr_fill")
    return SparseRows(row_ptr, col_idx, values, rows, cols)


def mosaic_sparse_gather_rows(p: SparseRows, d: torch.Tensor, ncols: int, c: torch.Tensor,
                              subtract: bool = False) -> None:
    """c[i, :ncols] +-= sum_j P[i, j] d[j, :ncols] (P: rows x r sparse)."""
    _need(d, p.cols, ncols, "d", _INT, optional=False)
    _need(c, p.rows, ncols, "c", _INT, optional=False)
    _check(_lib.load().mosaic_sparse_gather_rows(p.rows, p.row_ptr.data_ptr(), p.col_idx.data_ptr(),
                                                 p.values.data_ptr(), d.data_ptr(), d.stride(0), ncols,
                                                 c.data_ptr(), c.stride(0), 1 if subtract else 0, _stream()),
           "mosaic_sparse_gather_rows")


def mosaic_sparse_stream_gather_rows(r: _lib.MosaicRng, rows: int, rcols: int, d: torch.Tensor, ncols: int,
                                     c: torch.Tensor, subtract: bool = False) -> None:
    """c[i, :ncols] +-= sum_j P[i, j] d[j, :ncols], P the rows x rcols SPARSE
    stream matrix of ``r`` (drawn inside the call)."""
    _need(d, rcols, ncols, "d", _INT, optional=False)
    _need(c, rows, ncols, "c", _INT, optional=False)
    _check(_lib.load().mosaic_sparse_stream_gather_rows(ctypes.byref(r), rows, rcols, d.data_ptr(), d.stride(0), ncols,
                                                        c.data_ptr(), c.stride(0), 1 if subtract else 0, _stream()),
           "mosaic_sparse_stream_gather_rows")


def mosaic_sparse_gather_cols(p: SparseRows, d: torch.Tensor, M: int, c: torch.Tensor,
                              subtract: bool = False, y_f32: Optional[torch.Tensor] = None,
                              s_rows: Optional[torch.Tensor] = None, s_cols: Optional[torch.Tensor] = None,
                              bias: Optional[torch.Tensor] = None) -> None:
    """c[m, n] +-= sum_j d[m, j] P[n, j] for m < M, n < P.rows; with y_f32,
    also y_f32 = c s_rows[m] s_cols[n] (+ bias[n]) of the finished c."""
    N = p.rows
    _need(d, M, p.cols, "d", _INT, optional=False)
    _need(c, M, N, "c", _INT, optional=False)
    _need(y_f32, M, N, "y_f32", (torch.float32,))
    if y_f32 is not None:
        _need(s_rows, 1, M, "s_rows", (torch.float32,), optional=False)
        _need(s_cols, 1, N, "s_cols", (torch.float32,), optional=False)
    _need(bias, 1, N, "bias", (torch.float32,))
    _check(_lib.load().mosaic_sparse_gather_cols(M, N, p.row_ptr.data_ptr(), p.col_idx.data_ptr(),
                                                 p.values.data_ptr(), d.data_ptr(), d.stride(0), c.data_ptr(),
                                                 c.stride(0), 1 if subtract else 0, _ptr(s_rows), _ptr(s_cols),
                                                 _ptr(bias), _ptr(y_f32), y_f32.stride(0) if y_f32 is not None else 0,
                                                 _stream()),
           "mosaic_sparse_gather_cols")


def mosaic_count_mismatches(a: torch.Tensor, b: torch.Tensor, count: torch.Tensor) -> None:
    """count[0] = number of entries where the int32 matrices a and b differ
    (same shape; count is a one-element int64 device tensor)."""
    if a.shape != b.shape or a.dim() != 2:
        raise ValueError("a and b must be matrices of the same shape")
    if count.dtype != torch.int64 or count.numel() < 1:
        raise ValueError("count must be an int64 tensor")
    rows, cols = a.shape
    _check(_lib.load().mosaic_count_mismatches(a.data_ptr(), a.stride(0), b.data_ptr(), b.stride(0), rows, cols,
                                               count.data_ptr(), _stream()), "mosaic_count_mismatches")


def mosaic_sample_signs(r: _lib.MosaicRng, n: int, out: torch.Tensor) -> None:
    _need(out, 1, n, "out", (torch.int8,), optional=False)
    _check(_lib.load().mosaic_sample_signs(ctypes.byref(r), n, out.data_ptr(), _stream()), "mosaic_sample_signs")


def mosaic_hadamard_rotate(x: torch.Tensor, y: torch.Tensor, block: Optional[int] = None,
                           signs: Optional[torch.Tensor] = None, inverse: bool = False) -> None:
    rows, n = x.shape
    _need(x, rows, n, "x", (torch.float32,), optional=False)
    _need(y, rows, n, "y", (torch.float32,), optional=False)
    _need(signs, 1, n, "signs", (torch.int8,))
    _check(_lib.load().mosaic_hadamard_rotate(x.data_ptr(), x.stride(0), y.data_ptr(), y.stride(0), rows, n,
                                              n if block is None else block, _ptr(signs), 1 if inverse else 0,
                                              _stream()), "mosaic_hadamard_rotate")


def mosaic_hadamard28_rotate(x: torch.Tensor, y: torch.Tensor, signs: Optional[torch.Tensor] = None,
                             inverse: bool = False) -> None:
    rows, n = x.shape
    _need(x, rows, n, "x", (torch.float32,), optional=False)
    _need(y, rows, n, "y", (torch.float32,), optional=False)
    _need(signs, 1, n, "signs", (torch.int8,))
    _check(_lib.load().mosaic_hadamard28_rotate(x.data_ptr(), x.stride(0), y.data_ptr(), y.stride(0), rows, n,
                                                _ptr(signs), 1 if inverse else 0, _stream()),
           "mosaic_hadamard28_rotate")


def mosaic_quantize_rows(x: torch.Tensor, qmax: int, q: Optional[torch.Tensor] = None,
                         q_dig: Optional[Digits] = None, scale: Optional[torch.Tensor] = None) -> None:
    rows, n = x.shape
    _need(x, rows, n, "x", (torch.float32,), optional=False)
    _need(q, rows, n, "q", _INT)
    _need_dig(q_dig, rows, n, "q_dig")
    _need(scale, 1, rows, "scale", (torch.float32,))
    _check(_lib.load().mosaic_quantize_rows(x.data_ptr(), x.stride(0), rows, n, qmax, _ptr(q),
                                            q.stride(0) if q is not None else 0,
                                            q_dig.ptr if q_dig else None, q_dig.pitch if q_dig else 0,
                                            _ptr(scale), _stream()), "mosaic_quantize_rows")


def mosaic_probe_mfma_i8(mode: int, iters: int, out: torch.Tensor) -> int:
    """Launches the register-only MFMA probe (measurement aid); returns the
    int8 operations launched. ``out`` is a one-element int32 device tensor."""
    ops = ctypes.c_int64(0)
    _check(_lib.load().mosaic_probe_mfma_i8(mode, iters, out.data_ptr(), ctypes.byref(ops), _stream()),
           "mosaic_probe_mfma_i8")
    return int(ops.value)
