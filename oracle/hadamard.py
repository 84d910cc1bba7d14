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


# ---------------------------------------------------------------------------
# The order-28 Hadamard matrix and the rotation H_28 (x) H_b for n = 28 b
# ---------------------------------------------------------------------------
# 28672 = 28 x 1024 is not a power of two. The block-diagonal rotation above
# mixes entries only within blocks of b; H_28 (x) H_b mixes all n. A
# Hadamard matrix of order 28 comes from Paley's first construction, which
# gives one of order q + 1 for every prime power q = 3 (mod 4); here
# q = 27 = 3^3 (a reading: any Hadamard matrix of order 28 would do, this is
# the one built here).

def gf27_mul(a: int, b: int) -> int:
    """Product in GF(27) = GF(3)[t] / (t^3 + 2 t + 1): an element c0 + 3 c1 +
    9 c2 stands for c0 + c1 t + c2 t^2 (c_i in GF(3)); t^3 reduces to t + 2."""
    pa = [a % 3, (a // 3) % 3, a // 9]
    pb = [b % 3, (b // 3) % 3, b // 9]
    prod = [0] * 5
    for i in range(3):
        for j in range(3):
            prod[i + j] += pa[i] * pb[j]
    for k in (4, 3):                      # t^k = t^(k-3) (t + 2)
        c = prod[k]
        prod[k] = 0
        prod[k - 2] += c
        prod[k - 3] += 2 * c
    return (prod[0] % 3) + 3 * (prod[1] % 3) + 9 * (prod[2] % 3)


def gf27_sub(a: int, b: int) -> int:
    return ((a % 3 - b % 3) % 3) + 3 * (((a // 3) % 3 - (b // 3) % 3) % 3) + 9 * ((a // 9 - b // 9) % 3)


def gf27_quadratic_character() -> np.ndarray:
    """chi(a): 0 for a = 0, +1 for the non-zero squares, -1 otherwise."""
    squares = {gf27_mul(a, a) for a in range(1, 27)}
    return np.array([0] + [1 if a in squares else -1 for a in range(1, 27)], dtype=np.int64)


def paley_hadamard_28() -> np.ndarray:
    """H = I + S with S = [[0, 1^T], [-1, Q]], Q[i][j] = chi(e_i - e_j) the
    Jacobsthal matrix of GF(27) (elements in index order). Since 27 = 3 (mod
    4), chi(-1) = -1, Q is skew-symmetric and Q Q^T = 27 I - J, so
    H H^T = 28 I."""
    chi = gf27_quadratic_character()
    Q = np.array([[chi[gf27_sub(i, j)] for j in range(27)] for i in range(27)], dtype=np.int64)
    S = np.zeros((28, 28), dtype=np.int64)
    S[0, 1:] = 1
    S[1:, 0] = -1
    S[1:, 1:] = Q
    return np.eye(28, dtype=np.int64) + S


def rotate_kron28(x: np.ndarray, signs: np.ndarray, inverse: bool = False) -> np.ndarray:
    """Row-wise rotation by (H_28 (x) H_b) / sqrt(n), n = 28 b, b a power of
    two: entry i b + j of a row is entry j of block i. Forward: that matrix
    times d * x; inverse (its transpose): d * ((H_28^T (x) H_b) x) / sqrt(n)."""
    x = np.asarray(x, dtype=np.float64)
    rows, n = x.shape
    if n % 28:
        raise ValueError("n must be 28 b")
    b = n // 28
    H28 = paley_hadamard_28().astype(np.float64)
    d = np.asarray(signs, dtype=np.float64).reshape(1, n)
    v = (x * d if not inverse else x).reshape(rows, 28, b)
    v = fwht_unnormalised(v)                                  # H_b within every block
    v = np.einsum("ik,rkj->rij", H28.T if inverse else H28, v)   # H_28 across the blocks
    y = v.reshape(rows, n) / np.sqrt(n)
    return y * d if inverse else y
