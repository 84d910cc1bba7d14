"""Random Hadamard rotation (Section 5, "Random Hadamard rotation"; protocol
Pi_Sec-Linear, Init W step 1 and online step 1) in float64.

R = H D with H the normalised Walsh-Hadamard matrix (H H^T = I) and
D = diag(d), d in {+1, -1}^n. Activations are rotated as x -> R x and weights
as w -> w R^T; both are row operations in the build's row-major layout
(a token's feature vector, a weight row), so the kernel maps each row v to

    forward:  H (d * v)          inverse (R^T):  d * (H v)

H is taken in Sylvester (natural) order, H_n[i][j] = (-1)^popcount(i & j) / sqrt(n),
and applied with Fino's fast transform (Section 5 cites it for the O(n log n)
cost): log2(n) stages of butterflies (a, b) -> (a + b, a - b) followed by the
1/sqrt(n) scale.

Lengths that are not a power of two (a reading: the paper assumes the FWHT
applies) use the block-diagonal rotation I_{n/b} (x) H_b with one length-n
sign vector; it is orthogonal, so the product-preservation and norm-
preservation properties of the rotation still hold.
"""
from __future__ import annotations

import numpy as np


def fwht_unnormalised(x: np.ndarray) -> np.ndarray:
    """Fino's butterfly transform along the last axis (length a power of two),
    returning H_n x with entries +-1 (no scaling)."""
    y = np.array(x, dtype=np.float64, copy=True)
    n = y.shape[-1]
    if n & (n - 1):
        raise ValueError("length must be a power of two")
    lead = y.shape[:-1]
    h = 1
    while h < n:
        z = y.reshape(lead + (n // (2 * h), 2, h))
        a = z[..., 0, :].copy()
        b = z[..., 1, :].copy()
        z[..., 0, :] = a + b
        z[..., 1, :] = a - b
        y = z.reshape(lead + (n,))
        h *= 2
    return y


def sylvester_matrix(n: int) -> np.ndarray:
    """H_n with entries (-1)^popcount(i & j) (unnormalised), by its definition."""
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    pc = np.vectorize(lambda v: bin(int(v)).count("1"))(i & j)
    return np.where(pc % 2 == 0, 1.0, -1.0)


def rotate(x: np.ndarray, signs: np.ndarray, block: int | None = None,
           inverse: bool = False) -> np.ndarray:
    """Row-wise random Hadamard rotation of ``x`` (rows x n) in float64."""
    x = np.asarray(x, dtype=np.float64)
    rows, n = x.shape
    b = n if block is None else block
    if n % b:
        raise ValueError("n must be a multiple of the block length")
    d = np.asarray(signs, dtype=np.float64).reshape(1, n)
    scale = 1.0 / np.sqrt(b)
    if not inverse:
        v = (x * d).reshape(rows, n // b, b)
        return (fwht_unnormalised(v) * scale).reshape(rows, n)
    v = x.reshape(rows, n // b, b)
    return (fwht_unnormalised(v) * scale).reshape(rows, n) * d
