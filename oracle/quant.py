"""Fixed-point quantisation of Pi_Sec-Linear (Section 5 protocol box, Init W
step 2 and online step 1; "Straw-man solution" paragraph).

Each row v (a weight row, or a token's rotated activation) gets the scale
s = ||v||_inf / q_max and the code round(v / s) in [-q_max, q_max]; the
integer product is dequantised as s_w * s_x * Y.

Readings: rounding is to nearest with ties to even; an all-zero row takes
s = 1 (its codes are 0 either way). Where the decision is an integer code the
arithmetic is float32 on both sides (scale = fp32 division, code = fp32
division then round), as in the kernel; dequantisation is float64 here.

Window (same paragraph): an inner product of n codes bounded by q_w and q_x
stays inside the signed ring range when n * q_w * q_x <= 2^31 - 1.
"""
from __future__ import annotations

import numpy as np


def quantize_rows(x: np.ndarray, qmax: int):
    x = np.asarray(x, dtype=np.float32)
    amax = np.max(np.abs(x), axis=1)
    s = np.where(amax > 0, amax / np.float32(qmax), np.float32(1.0)).astype(np.float32)
    q = np.rint(x / s[:, None]).astype(np.int64)
    return q.astype(np.int32), s


def dequantize(y_int: np.ndarray, s_rows: np.ndarray, s_cols: np.ndarray) -> np.ndarray:
    return np.asarray(y_int, dtype=np.float64) * np.asarray(s_rows, np.float64)[:, None] \
        * np.asarray(s_cols, np.float64)[None, :]


def max_qx(n: int, q_w: int, margin: int = 0) -> int:
    """Largest q_x with n * (q_w + margin) * (q_x + margin) <= 2^31 - 1."""
    lim = (2 ** 31 - 1) // (n * (q_w + margin))
    return int(lim - margin)
