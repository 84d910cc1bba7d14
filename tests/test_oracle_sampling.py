"""Pins for the oracle's samplers (CPU only)."""
import math

import numpy as np
import pytest

from oracle import sampling as smp


def _poisson_dual_Z(sigma):
    """sum_{j in Z} exp(-j^2 / (2 sigma^2)) via Poisson summation:
    sigma sqrt(2 pi) sum_{k in Z} exp(-2 pi^2 sigma^2 k^2)."""
    s = 1.0
    for k in range(1, 50):
        s += 2 * math.exp(-2 * math.pi ** 2 * sigma ** 2 * k ** 2)
    return sigma * math.sqrt(2 * math.pi) * s


@pytest.mark.parametrize("sigma,bound", [(0.5, 4), (1.0, 8), (1.5, 12), (2.0, 16)])
def test_dgauss_thresholds_shape(sigma, bound):
    th = smp.dgauss_thresholds(sigma, bound)
    assert len(th) == 2 * bound
    assert all(0 <= a <= b <= 2 ** 32 for a, b in zip(th, th[1:]))
    counts = np.diff([0] + th + [2 ** 32])              # 2^32 * p_j, j = -B..B
    # symmetry p_j = p_{-j}
    assert np.all(np.abs(counts - counts[::-1]) <= 1)
    # central mass 1 / Z, with Z from the dual series (truncation of the
    # support at B changes Z by far less than a count)
    z = _poisson_dual_Z(sigma)
    assert abs(counts[bound] - 2 ** 32 / z) <= 1.5
    # ratio of neighbours p_{j+1} / p_j = exp(-(2j+1) / (2 sigma^2))
    for j in range(0, 3):
        a, b = counts[bound + j], counts[bound + j + 1]
        if b > 10 ** 5:
            assert abs(b / a - math.exp(-(2 * j + 1) / (2 * sigma ** 2))) < 5e-5


def test_dgauss_sigma_half_probabilities():
    """sigma = 0.5, bound 4: P(0) ~ 0.78657, P(+-1) ~ 0.10645, P(+-2) ~ 2.64e-4,
    P(+-3) ~ 1.2e-8, P(+-4) < 2^-32 (from exp(-j^2 * 2) / Z)."""
    counts = np.diff([0] + smp.dgauss_thresholds(0.5, 4) + [2 ** 32]) / 2 ** 32
    assert abs(counts[4] - 0.78657) < 1e-5
    assert abs(counts[5] - 0.10645) < 1e-5
    assert abs(counts[6] - 2.64e-4) < 1e-6
    assert 0 < counts[7] < 2e-8
    assert counts[8] == 0


def test_dgauss_zero_sigma_is_zero():
    m = smp.sample_matrix("dgauss", 4, 8, 1, 2, 3, sigma=0.0, bound=4)
    assert np.all(m == 0)


def test_dgauss_samples_match_distribution():
    m = smp.sample_matrix("dgauss", 512, 2048, 5, smp.STREAM_EW, 0, sigma=0.5, bound=4)
    v = m.view(np.int32).ravel()
    assert v.min() >= -3 and v.max() <= 3
    p = np.diff([0] + smp.dgauss_thresholds(0.5, 4) + [2 ** 32]) / 2 ** 32
    for j in (-2, -1, 0, 1, 2):
        f = np.mean(v == j)
        sd = math.sqrt(p[j + 4] * (1 - p[j + 4]) / v.size)
        assert abs(f - p[j + 4]) < 5 * sd + 1e-9
    assert abs(v.mean()) < 5 * math.sqrt(0.215 / v.size)
    var_ref = float(sum((j ** 2) * p[j + 4] for j in range(-4, 5)))
    assert abs(v.var() - var_ref) < 0.01


def test_dgauss_element_is_function_of_its_word():
    """Element e of a dgauss matrix is determined by word e of its stream
    (-B + number of thresholds <= that word)."""
    m = smp.sample_matrix("dgauss", 3, 7, 11, 0x50, 2, sigma=0.5, bound=4).view(np.int32).ravel()
    w = smp.stream_words(11, 0x50, 2, 0, 21)
    th = smp.dgauss_thresholds(0.5, 4)
    for e in range(21):
        assert m[e] == -4 + sum(int(w[e]) >= t for t in th)


def test_sparse_density_and_values():
    m = smp.sample_matrix("sparse", 1024, 1024, 3, smp.STREAM_S + 2, 0, log2_inv_density=6)
    nz = m != 0
    frac = nz.mean()
    sd = math.sqrt((1 / 64) * (63 / 64) / m.size)
    assert abs(frac - 1 / 64) < 5 * sd
    # element e uses gate word 2e and value word 2e+1
    w = smp.stream_words(3, smp.STREAM_S + 2, 0, 0, 2 * 64)
    flat = m.ravel()[:64]
    for e in range(64):
        exp = w[2 * e + 1] if (w[2 * e] >> 26) == 0 else 0
        assert flat[e] == exp
    vals = m[nz].astype(np.uint64)
    assert abs(vals.mean() / 2 ** 32 - 0.5) < 0.02


def test_uniform_is_raw_words():
    m = smp.sample_matrix("uniform", 5, 9, 17, 0x11, 4)
    assert np.array_equal(m.ravel(), smp.stream_words(17, 0x11, 4, 0, 45))


def test_signs_balanced():
    d = smp.sample_signs(1 << 16, 3)
    assert set(np.unique(d)) == {-1, 1}
    assert abs(d.mean()) < 5 / math.sqrt(d.size)
