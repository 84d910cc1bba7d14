"""Pins for the oracle's random Hadamard rotation (CPU only)."""
import json
import math
import os

import numpy as np
import pytest
import scipy.linalg

from oracle.hadamard import (fwht_unnormalised, gf27_mul, gf27_quadratic_character, gf27_sub, paley_hadamard_28,
                             rotate, rotate_kron28, sylvester_matrix)
from oracle.sampling import sample_signs
from synthetic_inputs import outlier_activations

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")


@pytest.mark.parametrize("n", [1, 2, 4, 8, 64, 512, 1024])
def test_fwht_matches_library_hadamard(n):
    rng = np.random.default_rng(n)
    x = rng.standard_normal((3, n))
    H = scipy.linalg.hadamard(n).astype(np.float64)
    assert np.allclose(fwht_unnormalised(x), x @ H.T, rtol=0, atol=1e-9 * n)


@pytest.mark.parametrize("n", [2, 16, 128])
def test_sylvester_definition(n):
    H = sylvester_matrix(n)
    assert np.array_equal(H, scipy.linalg.hadamard(n))
    assert np.array_equal(H @ H.T, n * np.eye(n))


def test_fwht_exact_on_small_integers():
    rng = np.random.default_rng(1)
    x = rng.integers(-1000, 1000, (4, 256)).astype(np.float64)
    H = sylvester_matrix(256)
    assert np.array_equal(fwht_unnormalised(x), x @ H.T)


def test_rotation_orthogonal_roundtrip_and_product():
    rng = np.random.default_rng(2)
    n = 512
    d = sample_signs(n, 3)
    x = rng.standard_normal((8, n))
    w = rng.standard_normal((5, n))
    rx = rotate(x, d)
    assert np.allclose(np.linalg.norm(rx, axis=1), np.linalg.norm(x, axis=1), rtol=1e-12)
    assert np.allclose(rotate(rx, d, inverse=True), x, atol=1e-12)
    # product preservation: (W R^T)(R X) = W X, with rows of both rotated by R
    assert np.allclose(rotate(w, d) @ rx.T, w @ x.T, atol=1e-10)
    # the rotation matrix itself: R = H D / sqrt(n)
    R = sylvester_matrix(n) @ np.diag(d.astype(np.float64)) / math.sqrt(n)
    assert np.allclose(rx, x @ R.T, atol=1e-12)


def test_block_diagonal_rotation():
    rng = np.random.default_rng(3)
    n, b = 7 * 64, 64
    d = sample_signs(n, 4)
    x = rng.standard_normal((3, n))
    y = rotate(x, d, block=b)
    for blk in range(n // b):
        s = slice(blk * b, (blk + 1) * b)
        assert np.allclose(y[:, s], rotate(x[:, s], d[s]), atol=1e-12)
    assert np.allclose(rotate(y, d, block=b, inverse=True), x, atol=1e-12)


def test_outlier_peak_to_rms_reduction():
    """Section 5 / appendix eq. had-inf-norm-bound: after rotation the peak of
    a row is of order ||x||_2 sqrt(log n / n), i.e. its max/RMS ratio is of
    order sqrt(log n). Outlier rows (N(0,1) with 0.1% entries x50) drop from
    a ratio in the tens to a few units."""
    n = 8192
    x = outlier_activations(64, n, seed=3)
    d = sample_signs(n, 3)
    y = rotate(x, d)

    def ratio(v):
        return np.max(np.abs(v), axis=1) / np.sqrt(np.mean(v ** 2, axis=1))
    before, after = ratio(x.astype(np.float64)), ratio(y)
    assert np.median(before) > 20
    assert np.all(after < math.sqrt(2 * math.log(2 * n)) + 1.0)
    assert np.median(after) < 5


def test_variance_reduction_figure():
    """n / log n at n = 4096 is about 340 (log taken base 2)."""
    with open(GOLDEN) as f:
        g = json.load(f)["variance_reduction_n4096"]
    assert abs(4096 / math.log2(4096) - g["value"]) <= g["tolerance"]


def test_gf27_is_a_field():
    """GF(3)[t] / (t^3 + 2 t + 1): the modulus has no root in GF(3) (so it is
    irreducible, being cubic); the multiplicative group of the 26 non-zero
    elements is cyclic-order compatible (a^26 = 1), every non-zero element
    has exactly one inverse, the product is associative and distributes
    over subtraction; 13 non-zero squares and chi(-1) = -1 (27 = 3 mod 4)."""
    assert all((r ** 3 + 2 * r + 1) % 3 != 0 for r in range(3))
    for a in range(1, 27):
        p = 1
        for _ in range(26):
            p = gf27_mul(p, a)
        assert p == 1
        assert sum(gf27_mul(a, b) == 1 for b in range(1, 27)) == 1
    rng = np.random.default_rng(27)
    for a, b, c in rng.integers(0, 27, (200, 3)):
        assert gf27_mul(gf27_mul(a, b), c) == gf27_mul(a, gf27_mul(b, c))
        assert gf27_mul(a, gf27_sub(b, c)) == gf27_sub(gf27_mul(a, b), gf27_mul(a, c))
    chi = gf27_quadratic_character()
    assert (chi == 1).sum() == 13 and (chi == -1).sum() == 13
    assert chi[gf27_sub(0, 1)] == -1


def test_paley_28_is_a_hadamard_matrix():
    """Entries +-1 and H H^T = 28 I exactly; H = I + S with S skew-symmetric
    (a skew-Hadamard matrix, as Paley's first construction gives)."""
    H = paley_hadamard_28()
    assert set(np.unique(H)) == {-1, 1}
    assert np.array_equal(H @ H.T, 28 * np.eye(28, dtype=np.int64))
    S = H - np.eye(28, dtype=np.int64)
    assert np.array_equal(S, -S.T)


@pytest.mark.parametrize("b", [4, 16])
def test_kron28_rotation_matches_explicit_kronecker(b):
    """The row rotation equals the explicit matrix (H_28 (x) H_b) / sqrt(28 b)
    (numpy's Kronecker product, scipy's Sylvester H_b) applied to d * x, and
    its inverse applies the transpose and then d."""
    n = 28 * b
    rng = np.random.default_rng(b)
    x = rng.standard_normal((3, n))
    d = np.where(rng.random(n) < 0.5, -1.0, 1.0)
    K = np.kron(paley_hadamard_28().astype(np.float64), scipy.linalg.hadamard(b).astype(np.float64)) / math.sqrt(n)
    assert np.allclose(rotate_kron28(x, d), (K @ (x * d).T).T, atol=1e-12)
    assert np.allclose(rotate_kron28(x, d, inverse=True), (K.T @ x.T).T * d, atol=1e-12)


def test_kron28_roundtrip_norm_and_outliers():
    """n = 28672 = 28 x 1024: orthogonal (round trip, norms), and on outlier
    rows the peak-to-RMS ratio falls at least as far as with the
    block-diagonal rotation I_28 (x) H_1024, which mixes only within blocks."""
    n = 28672
    x = outlier_activations(16, n, seed=5)
    d = sample_signs(n, 5)
    y = rotate_kron28(x, d)
    assert np.allclose(rotate_kron28(y, d, inverse=True), x, atol=1e-9)
    assert np.allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x.astype(np.float64), axis=1), rtol=1e-12)

    def ratio(v):
        return np.max(np.abs(v), axis=1) / np.sqrt(np.mean(v ** 2, axis=1))
    kron, blockdiag = ratio(y), ratio(rotate(x, d, block=1024))
    assert np.median(kron) <= np.median(blockdiag) + 1e-9
    assert np.all(kron < math.sqrt(2 * math.log(2 * n)) + 1.0)
