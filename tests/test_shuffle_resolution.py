"""Host check of the closed form the fixed-weight (WEIGHT) row kernels use to
find a partial Fisher-Yates shuffle's columns without running its swaps in
order (Example 4.1 rows of weight t; reading R27): a model of the kernel's
steps -- a table over positions counting each position's choosers and
keeping the first one to arrive (arrival order random, as for the LDS
atomics), a list of the steps on positions chosen more than once, and the
chains through both -- against the swaps themselves, on random rows
including full permutations (t = r) where nearly every position is chosen
twice. The kernels' outputs are compared with the oracle's shuffle in
test_gpu_sparse.py; this pins the argument the fast form rests on."""
import numpy as np
import pytest


def _swaps(ks, cols):
    perm = list(range(cols))
    out = []
    for j, k in enumerate(ks):
        perm[j], perm[k] = perm[k], perm[j]
        out.append(perm[j])
    return out


def _table_form(ks, cols, rng):
    t = len(ks)
    tab = [0] * cols
    for j in rng.permutation(t):                  # atomics land in any order
        old = tab[ks[j]]
        tab[ks[j]] = old + 0x10000
        if (old >> 16) == 0:
            tab[ks[j]] |= int(j)
    several = [j for j in range(t) if (tab[ks[j]] >> 16) >= 2]
    rng.shuffle(several)                          # the list's order is arbitrary too

    def latest(p, before):
        e = tab[p]
        if (e >> 16) == 0:
            return -1
        if (e >> 16) == 1:
            return (e & 0xFFFF) if (e & 0xFFFF) < before else -1
        return max([i for i in several if i < before and ks[i] == p], default=-1)

    out = []
    for j in range(t):
        x = latest(ks[j], j)
        col = ks[j]
        if x >= 0:
            y = latest(x, x)
            while y >= 0:
                x, y = y, latest(y, y)
            col = x
        out.append(col)
    return out


@pytest.mark.parametrize("t,cols", [(80, 1024), (80, 652), (80, 80), (256, 256), (256, 300), (65, 65),
                                    (1, 1), (0, 7), (200, 210), (256, 8192)])
def test_table_form_matches_swaps(t, cols):
    rng = np.random.default_rng(1000 * t + cols)
    for _ in range(40):
        u = rng.integers(0, 2 ** 32, t, dtype=np.uint64)
        ks = [j + ((int(u[j]) * (cols - j)) >> 32) for j in range(t)]
        assert all(j <= k < cols for j, k in enumerate(ks))
        assert _table_form(ks, cols, rng) == _swaps(ks, cols)
