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


# --- fixed-weight LPN noise (Example 4.1: t nonzeros per noise vector) ---

def test_weighted_rows_exact_weight_and_range():
    """Every row has exactly t distinct columns in [0, cols) (also t = cols,
    a full permutation, and t = 0)."""
    for cols, t in [(1536, 80), (1024, 80), (7, 7), (64, 1), (33, 0)]:
        pos, val = smp.weighted_rows(range(200), cols, t, 11, 0x44, 2)
        assert pos.shape == (200, t) and val.shape == (200, t)
        for row in pos:
            assert len(set(row.tolist())) == t
            assert all(0 <= p < cols for p in row)
        if t == cols:
            assert all(sorted(row.tolist()) == list(range(cols)) for row in pos)
    S = smp.sample_matrix("weight", 300, 1536, 5, 0x43, 1, row_weight=80)
    assert np.all(np.count_nonzero(S, axis=1) == 80)     # a zero value has probability 80 * 2^-32


def test_weighted_subsets_uniform():
    """All C(5, 2) = 10 column pairs (and all 4! orders of a full shuffle of
    4) appear equally often: a partial shuffle that picked from the wrong
    range or swapped the wrong entries biases these counts."""
    pos, _ = smp.weighted_rows(range(30000), 5, 2, 3, 0x45, 0)
    keys = np.sort(pos, axis=1)
    codes = keys[:, 0] * 5 + keys[:, 1]
    counts = np.bincount(codes, minlength=25)
    cells = counts[[a * 5 + b for a in range(5) for b in range(a + 1, 5)]]
    assert cells.sum() == 30000
    exp = 3000.0
    assert float(((cells - exp) ** 2 / exp).sum()) < 33.7          # chi2, 9 dof, p ~ 1e-4
    perm, _ = smp.weighted_rows(range(24000), 4, 4, 4, 0x46, 0)
    codes = perm[:, 0] * 64 + perm[:, 1] * 16 + perm[:, 2] * 4 + perm[:, 3]
    _, counts = np.unique(codes, return_counts=True)
    assert counts.size == 24
    assert float(((counts - 1000.0) ** 2 / 1000.0).sum()) < 49.7     # chi2, 23 dof, p ~ 1e-3


def test_weighted_positions_uniform_at_paper_size():
    """At r = 1536, t = 80 each column is chosen with probability t / r."""
    pos, val = smp.weighted_rows(range(3000), 1536, 80, 8, 0x47, 0)
    counts = np.bincount(pos.ravel(), minlength=1536)
    exp = 3000 * 80 / 1536
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert abs(chi2 - 1535) < 6 * math.sqrt(2 * 1535)
    by = np.frombuffer(val.tobytes(), dtype=np.uint8)
    bc = np.bincount(by, minlength=256)
    assert float(((bc - by.size / 256) ** 2 / (by.size / 256)).sum()) < 400


def test_weighted_row_uses_its_own_words():
    """Row i is a function of words 2 t i .. 2 t i + 2 t - 1 only: the same row
    drawn alone or inside a range agrees, and the first step's column is
    floor(u_0 cols / 2^32)."""
    t, cols = 80, 1024
    a, va = smp.weighted_rows([17], cols, t, 9, 0x48, 3)
    b, vb = smp.weighted_rows(range(10, 30), cols, t, 9, 0x48, 3)
    assert np.array_equal(a[0], b[7]) and np.array_equal(va[0], vb[7])
    w = smp.stream_words(9, 0x48, 3, 2 * t * 17, 2 * t)
    assert a[0, 0] == (int(w[0]) * cols) >> 32
    assert np.array_equal(va[0], w[1::2])
