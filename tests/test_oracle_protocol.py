"""Pins for the oracle's Pi_Sec-Approx-MatMul (CPU only).

The strongest pin is algebraic: expanding W'X' shows the unmasked result is
exactly (W + E_w)(X + E_x) over Z_{2^32}, for every depth and every mask draw
(Section 4.1 eq. approx-error; Section 4.2 "Unmasking"). It is checked here
against Python-integer arithmetic, which shares nothing with the oracle's
ring routines.
"""
import math

import numpy as np
import pytest

from oracle import protocol as proto
from oracle.ring import lift, ring_add, ring_matmul, ring_sub
from synthetic_inputs import NoiseSpec, ProtocolParams

SMALL = NoiseSpec("dgauss", 0.5, 4)
ZERO = NoiseSpec("zero", 0.0, 0)


def _int_matmul(a, b):
    """Python-integer matrix product, reduced mod 2^32."""
    a = [[int(v) for v in row] for row in np.asarray(a, dtype=np.uint32)]
    b = [[int(v) for v in row] for row in np.asarray(b, dtype=np.uint32)]
    n, k, m = len(a), len(b), len(b[0])
    return np.array([[sum(a[i][t] * b[t][j] for t in range(k)) % (1 << 32) for j in range(m)]
                     for i in range(n)], dtype=np.uint32)


def _plain(l, n, m, seed):
    rng = np.random.default_rng(seed)
    A = rng.integers(-127, 128, (l, n), dtype=np.int8)
    W = rng.integers(-127, 128, (m, n), dtype=np.int8)
    return A, W


@pytest.mark.parametrize("ranks", [(8,), (8, 4), (8, 6, 4)])
@pytest.mark.parametrize("noise", [SMALL, ZERO])
def test_unmask_equals_noisy_product_bruteforce(ranks, noise):
    A, W = _plain(5, 12, 10, seed=len(ranks))
    p = ProtocolParams(ranks=ranks, noise=noise, sparse_log2_inv_density=1)
    res = proto.run(A, W, p, seed=1234, weight_id=3, call_id=7)
    X = A.T.astype(np.int64)
    lhs = (W.astype(np.int64) + lift(res.ws.E_w).astype(np.int64))
    rhs = (X + lift(res.cs.E_x).astype(np.int64))
    expect = _int_matmul(lhs & 0xFFFFFFFF, rhs & 0xFFFFFFFF)
    assert np.array_equal(res.Y, expect)
    if noise.kind == "zero":
        assert np.array_equal(lift(res.Y).astype(np.int64), W.astype(np.int64) @ X)


@pytest.mark.parametrize("ranks", [(16,), (16, 8), (24, 16, 8)])
def test_mask_invariance_without_noise(ranks):
    """With E = 0 every mask draw (seed, ids) unmasks to exactly W X."""
    A, W = _plain(7, 40, 24, seed=9)
    p = ProtocolParams(ranks=ranks, noise=ZERO, sparse_log2_inv_density=2)
    ref = W.astype(np.int64) @ A.T.astype(np.int64)
    for seed, wid, cid in [(1, 0, 0), (2, 5, 1), (0xDEADBEEF, 1, 99)]:
        res = proto.run(A, W, p, seed=seed, weight_id=wid, call_id=cid)
        assert np.array_equal(lift(res.Y).astype(np.int64), ref)
        # and the server really saw masked operands
        assert not np.array_equal(res.ws.W_masked, res.ws.W)


def test_sparse_levels_are_used():
    """Depth 2 at density 1/2: S_2 and T_2 are non-zero and enter W' and X'."""
    A, W = _plain(6, 32, 16, seed=1)
    p = ProtocolParams(ranks=(16, 8), noise=ZERO, sparse_log2_inv_density=1)
    res = proto.run(A, W, p, seed=5)
    assert np.count_nonzero(res.ws.S[1]) > 0 and np.count_nonzero(res.cs.T[1]) > 0
    lowrank = ring_matmul(res.ws.L, res.ws.Mc[1])
    assert not np.array_equal(res.ws.U_w, ring_add(lowrank, res.ws.E_w))


def test_simplified_unmask_agrees_for_depth_one():
    """Section 4.1 removes LM(X + E_x) and (W'N)R; the result equals the full
    protocol's unmask for d = 1."""
    A, W = _plain(6, 20, 14, seed=2)
    p = ProtocolParams(ranks=(8,), noise=SMALL)
    res = proto.run(A, W, p, seed=77)
    X = A.T.astype(np.int64) & 0xFFFFFFFF
    XE = ring_add(X.astype(np.uint32), res.cs.E_x)
    LM = ring_matmul(res.ws.L, res.ws.M[0])
    WN = ring_matmul(res.ws.W_masked, res.ws.N[0])
    simple = ring_sub(ring_sub(res.Y_masked, ring_matmul(LM, XE)), ring_matmul(WN, res.cs.R))
    assert np.array_equal(simple, res.Y)


def test_masked_operands_look_uniform():
    A, W = _plain(64, 256, 128, seed=3)
    res = proto.run(A, W, ProtocolParams(ranks=(32,), noise=SMALL), seed=11)
    for mat in (res.ws.W_masked, res.X_masked):
        by = np.frombuffer(mat.tobytes(), dtype=np.uint8)
        c = np.bincount(by, minlength=256)
        e = by.size / 256
        assert float(((c - e) ** 2 / e).sum()) < 400


def test_error_bound_theorem():
    """Theorem 4.2: entry (j, k) of E_w X + W E_x + E_w E_x is sub-Gaussian with
    parameter sigma sqrt(||x_k||^2 + ||w_j||^2); the tail fraction above t
    such parameters stays below 2 exp(-t^2 / 2). Also mean zero (Lemma A.1)."""
    A, W = _plain(64, 512, 256, seed=4)
    res = proto.run(A, W, ProtocolParams(ranks=(64,), noise=SMALL), seed=21)
    X = A.T.astype(np.float64)
    err = lift(res.Y).astype(np.float64) - W.astype(np.float64) @ X
    xn = (X ** 2).sum(axis=0)
    wn = (W.astype(np.float64) ** 2).sum(axis=1)
    scale = 0.5 * np.sqrt(wn[:, None] + xn[None, :])
    z = np.abs(err) / scale
    for t in (1.5, 2.0, 3.0):
        assert np.mean(z > t) <= 2 * math.exp(-t * t / 2)
    assert abs(err.mean()) < 5 * err.std() / math.sqrt(err.size)
    # the cross term E_w E_x is small next to the other two
    cross = lift(res.ws.E_w).astype(np.float64) @ lift(res.cs.E_x).astype(np.float64)
    assert np.abs(cross).mean() < 0.05 * np.abs(err).mean()


def test_chain_shapes():
    p = ProtocolParams(ranks=(24, 16, 8), noise=ZERO)
    A, W = _plain(3, 40, 12, seed=5)
    res = proto.run(A, W, p, seed=1)
    assert [m.shape for m in res.ws.Mc] == [(24, 40), (16, 40), (8, 40)]
    assert [m.shape for m in res.ws.Nc] == [(40, 24), (40, 16), (40, 8)]
    assert [q.shape for q in res.Q] == [(24, 3), (16, 3), (8, 3)]
    assert res.ws.L.shape == (12, 8)
    assert res.ws.S[1].shape == (12, 24) and res.ws.S[2].shape == (12, 16)


@pytest.mark.parametrize("noise", [SMALL, ZERO])
def test_sampled_depth1_matches_full_run(noise):
    """The sampled routine (used at full sizes) restates the depth-1 protocol
    row by row; it must agree with the full oracle on every sampled output."""
    rng = np.random.default_rng(8)
    A = rng.integers(-127, 128, (20, 96), dtype=np.int8)
    W = rng.integers(-127, 128, (30, 96), dtype=np.int8)
    p = ProtocolParams(ranks=(64,), noise=noise)
    full = proto.run(A, W, p, 77, 2, 5)
    I, J = [0, 7, 19], [1, 29, 11]
    s = proto.sampled_depth1(A[I], W[J], I, J, 96, p, 77, 2, 5)
    assert np.array_equal(s["Y"], full.Y.T[np.ix_(I, J)])
    assert np.array_equal(s["Y_masked"], full.Y_masked.T[np.ix_(I, J)])
    assert np.array_equal(s["Q"], full.Q[0].T[I])
    assert np.array_equal(s["W_masked"], full.ws.W_masked[J])
    assert np.array_equal(s["A_masked"], full.X_masked.T[I])
    assert np.array_equal(s["K_c"], full.cs.K.T[np.ix_(I, J)])
    assert np.array_equal(s["Y"], s["identity"])


@pytest.mark.parametrize("weights", [(3,), (5, 2)])
def test_fixed_weight_levels(weights):
    """With fixed row weights (Example 4.1's parameterisation) S_{i+1} has t
    nonzeros in every row, T_{i+1} in every column (one token's noise
    vector), and unmasking still returns (W + E_w)(X + E_x) exactly."""
    ranks = (12, 8, 6)[: len(weights) + 1]
    A, W = _plain(5, 12, 10, seed=11)
    p = ProtocolParams(ranks=ranks, noise=SMALL, lpn_weights=weights)
    res = proto.run(A, W, p, seed=77, weight_id=1, call_id=2)
    for i, t in enumerate(weights, start=1):
        assert np.all(np.count_nonzero(res.ws.S[i], axis=1) == t)
        assert np.all(np.count_nonzero(res.cs.T[i], axis=0) == t)
    X = A.T.astype(np.int64)
    lhs = W.astype(np.int64) + lift(res.ws.E_w).astype(np.int64)
    rhs = X + lift(res.cs.E_x).astype(np.int64)
    assert np.array_equal(res.Y, _int_matmul(lhs & 0xFFFFFFFF, rhs & 0xFFFFFFFF))
