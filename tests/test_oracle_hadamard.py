"""Pins for the oracle's random Hadamard rotation (CPU only)."""
import json
import math
import os

import numpy as np
import pytest
import scipy.linalg

from oracle.hadamard import fwht_unnormalised, rotate, sylvester_matrix
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
