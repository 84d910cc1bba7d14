"""Pins for the oracle's integrity check (Freivalds' test, Appendix
"Computational integrity"; Section 4.2 box, Init W step 3, online step 4).

* honest outputs of the oracle protocol are accepted at depths 1-3;
* a corrupted output entry changes exactly one column of the right-hand side,
  by the closed form a[:, j] * delta (mod 2^32), computed here with Python
  integers;
* over Z_{2^32} a single vector misses an error delta with probability
  2^-(32 - v(delta)): never (in 400 trials) for odd delta, about half the
  time for delta = 2^31, about a quarter for delta = 3 * 2^30.
"""
import numpy as np
import pytest

from oracle import integrity as integ
from oracle import protocol as proto
from oracle.ring import ring_sub
from synthetic_inputs import NoiseSpec, ProtocolParams

SMALL = NoiseSpec("dgauss", 0.5, 4)
ZERO = NoiseSpec("zero", 0.0, 0)


def _run(ranks, noise, seed=5, shape=(6, 40, 24)):
    l, n, m = shape
    rng = np.random.default_rng(seed)
    A = rng.integers(-127, 128, (l, n), dtype=np.int8)
    W = rng.integers(-127, 128, (m, n), dtype=np.int8)
    p = ProtocolParams(ranks=ranks, noise=noise, sparse_log2_inv_density=2)
    return proto.run(A, W, p, seed=seed, weight_id=1, call_id=2)


def _check(res, t, seed=5, weight_id=1, Y_t=None, Q_t=None):
    ranks = [mc.shape[0] for mc in res.ws.Mc]
    aW, aQ = integ.check_vectors(t, res.ws.W.shape[0], ranks, seed, weight_id)
    cT = integ.key(aW, aQ, res.ws.W_masked, {i + 1: mc for i, mc in enumerate(res.ws.Mc)})
    Y_t = res.Y_masked.T.copy() if Y_t is None else Y_t
    Q_t = {i + 1: q.T.copy() for i, q in enumerate(res.Q)} if Q_t is None else Q_t
    return aW, aQ, integ.sides(cT, aW, aQ, res.X_masked.T, Y_t, Q_t)


@pytest.mark.parametrize("ranks", [(16,), (16, 8), (24, 16, 8)])
@pytest.mark.parametrize("noise", [SMALL, ZERO])
def test_honest_outputs_accepted(ranks, noise):
    res = _run(ranks, noise)
    _, _, (lhs, rhs) = _check(res, t=4)
    assert lhs.shape == (4, 6) and integ.accept(lhs, rhs)


def test_corruption_closed_form():
    res = _run((16, 8), SMALL)
    t, m0, j0, delta = 5, 3, 17, 0x12345
    Y_t = res.Y_masked.T.copy()
    Y_t[m0, j0] = np.uint32((int(Y_t[m0, j0]) + delta) % 2 ** 32)
    aW, aQ, (lhs, rhs) = _check(res, t, Y_t=Y_t)
    diff = ring_sub(rhs, lhs)
    expect = np.zeros_like(diff)
    for j in range(t):
        expect[j, m0] = (int(aW[j, j0]) * delta) % 2 ** 32
    assert np.array_equal(diff, expect)
    # a corrupted Q entry of level 2
    Q_t = {i + 1: q.T.copy() for i, q in enumerate(res.Q)}
    Q_t[2][1, 5] = np.uint32((int(Q_t[2][1, 5]) + 7) % 2 ** 32)
    aW, aQ, (lhs, rhs) = _check(res, t, Q_t=Q_t)
    diff = ring_sub(rhs, lhs)
    expect = np.zeros_like(diff)
    for j in range(t):
        expect[j, 1] = (int(aQ[2][j, 5]) * 7) % 2 ** 32
    assert np.array_equal(diff, expect)


@pytest.mark.parametrize("delta,lo,hi", [(1, 0, 0), (0x7FFF, 0, 0), (1 << 31, 150, 250), (3 << 30, 60, 140)])
def test_single_vector_soundness_over_the_ring(delta, lo, hi):
    """400 independent single-vector checks (fresh weight ids) of one output
    corrupted by delta: the number of misses follows Binomial(400, 2^-(32-v))."""
    res = _run((16,), SMALL, shape=(3, 24, 8))
    misses = 0
    for wid in range(400):
        aW, aQ = integ.check_vectors(1, 8, [16], 5, wid)
        cT = integ.key(aW, aQ, res.ws.W_masked, {1: res.ws.Mc[0]})
        Y_t = res.Y_masked.T.copy()
        Y_t[1, 2] = np.uint32((int(Y_t[1, 2]) + delta) % 2 ** 32)
        lhs, rhs = integ.sides(cT, aW, aQ, res.X_masked.T, Y_t, {1: res.Q[0].T.copy()})
        misses += integ.accept(lhs, rhs)
    assert lo <= misses <= hi, misses
