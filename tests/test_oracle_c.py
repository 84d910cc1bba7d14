"""Pins for the oracle's plain C leg (CPU only): the ring product against
Python-integer brute force and the numpy ring product, and the C rotation
against the Sylvester matrix and the numpy oracle."""
import numpy as np

from oracle import _cring
from oracle import hadamard as ohad
from oracle.ring import ring_matmul

EDGE = np.array([0, 1, 2, 255, 256, 2 ** 31 - 1, 2 ** 31, 2 ** 32 - 1, 0x80808080], dtype=np.uint64)


def test_ring_matmul_nt_bruteforce():
    rng = np.random.default_rng(3)
    for m, n, k in [(1, 1, 1), (3, 4, 7), (5, 2, 33)]:
        a = rng.choice(EDGE, size=(m, k)).astype(np.uint32)
        b = rng.integers(0, 2 ** 32, (n, k), dtype=np.uint64).astype(np.uint32)
        got = _cring.ring_matmul_nt(a, b)
        for i in range(m):
            for j in range(n):
                assert int(got[i, j]) == sum(int(a[i, t]) * int(b[j, t]) for t in range(k)) % (1 << 32)


def test_ring_matmul_nt_matches_numpy_ring():
    rng = np.random.default_rng(4)
    a = rng.integers(0, 2 ** 32, (70, 300), dtype=np.uint64).astype(np.uint32)
    b = rng.integers(0, 2 ** 32, (45, 300), dtype=np.uint64).astype(np.uint32)
    assert np.array_equal(_cring.ring_matmul_nt(a, b), ring_matmul(a, b.T))


def test_rotation_matches_matrix_and_inverts():
    rng = np.random.default_rng(5)
    n = 64
    x = rng.standard_normal((9, n))
    d = np.where(rng.integers(0, 2, n) == 0, 1, -1).astype(np.int8)
    H = ohad.sylvester_matrix(n) / np.sqrt(n)
    y = _cring.rotate_rows(x, d)
    assert np.allclose(y, (x * d) @ H.T, rtol=0, atol=1e-12)
    assert np.allclose(_cring.rotate_rows(y, d, inverse=True), x, rtol=0, atol=1e-12)
    big = rng.standard_normal((5, 8192))
    db = np.where(rng.integers(0, 2, 8192) == 0, 1, -1).astype(np.int8)
    assert np.allclose(_cring.rotate_rows(big, db), ohad.rotate(big, db), rtol=0, atol=1e-9)


def test_threads_positive():
    assert _cring.threads() >= 1


def test_depth1_c_call_matches_protocol():
    """The C-leg depth-1 call equals oracle.protocol.run (transposed to the
    build orientation) on every intermediate, and unmasks to the noisy
    product."""
    from oracle import protocol as proto
    from oracle.ring import lift
    from synthetic_inputs import PARAMS_D1_SMALL_R128, int8_operands
    A, W = int8_operands(64, 512, 200, 0)
    ref = proto.run(A, W, PARAMS_D1_SMALL_R128, 99, weight_id=2, call_id=5)
    w = proto.init_w_depth1_c(W, PARAMS_D1_SMALL_R128, 99, 2)
    got = proto.call_depth1_c(w, A, PARAMS_D1_SMALL_R128, 99, 5)
    assert np.array_equal(w.W_masked, ref.ws.W_masked)
    assert np.array_equal(got["A_masked"], ref.X_masked.T)
    assert np.array_equal(got["Y_masked"], ref.Y_masked.T)
    assert np.array_equal(got["Q"], ref.Q[0].T)
    assert np.array_equal(got["K_c"], ref.cs.K.T)
    assert np.array_equal(got["Y"], ref.Y.T)
    ident = (A.astype(np.int64) + lift(got["E_a"])) @ (W.astype(np.int64) + lift(ref.ws.E_w)).T
    assert np.array_equal(lift(got["Y"]).astype(np.int64), ident)
