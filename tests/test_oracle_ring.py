"""Pins for the oracle's ring arithmetic and signed-digit form (CPU only)."""
import json
import os

import numpy as np

from oracle.ring import (digit_layout_pad_is_zero, digit_layout_unpack, from_signed_digits,
                         lift, padded_k, ring_matmul, signed_digits, to_ring)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")
EDGE = [0, 1, 2, 127, 128, 255, 256, 2 ** 31 - 1, 2 ** 31, 2 ** 31 + 1, 2 ** 32 - 2, 2 ** 32 - 1,
        0x80808080, 0x7F7F7F7F, 0xFF00FF00, 0x00FF00FF]


def _brute_matmul(x, y):
    a, b = x.shape
    c = y.shape[1]
    out = np.zeros((a, c), dtype=np.uint32)
    for i in range(a):
        for j in range(c):
            s = 0
            for k in range(b):
                s += int(x[i, k]) * int(y[k, j])
            out[i, j] = s % (1 << 32)
    return out


def test_ring_matmul_bruteforce_edges():
    rng = np.random.default_rng(0)
    for shape in [(1, 1, 1), (3, 5, 2), (4, 16, 7), (6, 33, 5)]:
        a, b, c = shape
        x = rng.choice(np.array(EDGE, dtype=np.uint64), size=(a, b)).astype(np.uint32)
        y = rng.integers(0, 2 ** 32, size=(b, c), dtype=np.uint64).astype(np.uint32)
        y[0, :] = 2 ** 32 - 1
        assert np.array_equal(ring_matmul(x, y), _brute_matmul(x, y))


def test_ring_matmul_linearity_and_identity():
    rng = np.random.default_rng(1)
    x1 = rng.integers(0, 2 ** 32, (8, 20), dtype=np.uint64).astype(np.uint32)
    x2 = rng.integers(0, 2 ** 32, (8, 20), dtype=np.uint64).astype(np.uint32)
    y = rng.integers(0, 2 ** 32, (20, 6), dtype=np.uint64).astype(np.uint32)
    lhs = ring_matmul(((x1.astype(np.uint64) + x2) & 0xFFFFFFFF).astype(np.uint32), y)
    rhs = ((ring_matmul(x1, y).astype(np.uint64) + ring_matmul(x2, y)) & 0xFFFFFFFF).astype(np.uint32)
    assert np.array_equal(lhs, rhs)
    eye = np.eye(20, dtype=np.uint32)
    assert np.array_equal(ring_matmul(x1, eye), x1)


def test_int8_embedding_product_is_integer_product():
    """Sign-extended int8 operands: the ring product lifted to int32 is the
    integer product when it fits (n q^2 <= 2^31 - 1)."""
    rng = np.random.default_rng(2)
    a = rng.integers(-127, 128, (5, 300), dtype=np.int64)
    b = rng.integers(-127, 128, (300, 4), dtype=np.int64)
    assert np.array_equal(lift(ring_matmul(to_ring(a), to_ring(b))).astype(np.int64), a @ b)


def test_signed_digits_roundtrip_and_range():
    rng = np.random.default_rng(3)
    x = np.concatenate([np.array(EDGE, dtype=np.uint64),
                        rng.integers(0, 2 ** 32, 1 << 20, dtype=np.uint64)]).astype(np.uint32)
    d = signed_digits(x)
    assert d.dtype == np.int8 and d.shape == x.shape + (4,)
    assert np.array_equal(from_signed_digits(d), x)
    # every byte pattern of the four 8-bit positions in {0x00, 0x7f, 0x80, 0xff}
    vals = np.array([0x00, 0x7F, 0x80, 0xFF], dtype=np.uint32)
    combo = (vals[:, None, None, None] | (vals[None, :, None, None] << 8)
             | (vals[None, None, :, None] << 16) | (vals[None, None, None, :] << 24)).ravel()
    assert np.array_equal(from_signed_digits(signed_digits(combo)), combo)


def test_signed_digits_unique():
    """Distinct digit vectors in [-128, 127]^4 give distinct residues: check
    exhaustively that the low 16 bits determine digits 0 and 1 (the map of
    two digits to a residue mod 2^16 is a bijection)."""
    d0 = np.arange(-128, 128)[:, None]
    d1 = np.arange(-128, 128)[None, :]
    res = (d0 + 256 * d1) % (1 << 16)
    assert np.unique(res).size == 1 << 16


def test_ten_limb_products_reproduce_the_ring_product():
    """Only limb products with i + j <= 3 survive mod 2^32: their shifted sum
    equals a * b mod 2^32, and there are exactly ten of them."""
    with open(GOLDEN) as f:
        golden = json.load(f)
    pairs = [(i, j) for i in range(4) for j in range(4) if i + j <= 3]
    assert len(pairs) == golden["int8_products_per_int32_product"]["value"]
    rng = np.random.default_rng(4)
    a = np.concatenate([np.array(EDGE, dtype=np.uint64), rng.integers(0, 2 ** 32, 5000, dtype=np.uint64)])
    b = np.concatenate([np.array(EDGE[::-1], dtype=np.uint64), rng.integers(0, 2 ** 32, 5000, dtype=np.uint64)])
    da = signed_digits(a.astype(np.uint32)).astype(np.int64)
    db = signed_digits(b.astype(np.uint32)).astype(np.int64)
    acc = np.zeros(a.shape, dtype=object)
    for i, j in pairs:
        acc = acc + (da[:, i] * db[:, j]).astype(object) * (1 << (8 * (i + j)))
    got = np.array([int(v) % (1 << 32) for v in acc], dtype=np.uint64)
    ref = np.array([(int(p) * int(q)) % (1 << 32) for p, q in zip(a, b)], dtype=np.uint64)
    assert np.array_equal(got, ref)


def test_digit_layout_unpack():
    """Pack by the layout's definition with explicit loops; unpack restores."""
    rng = np.random.default_rng(5)
    for rows, K in [(1, 1), (3, 17), (2, 64), (5, 100)]:
        x = rng.integers(0, 2 ** 32, (rows, K), dtype=np.uint64).astype(np.uint32)
        Kp = padded_k(K)
        buf = np.zeros(rows * 4 * Kp, dtype=np.int8)
        for i in range(rows):
            for k in range(K):
                v = int(x[i, k])
                for t in range(4):
                    r = v & 0xFF
                    dig = r - 256 if r >= 128 else r
                    v = ((v - dig) >> 8) & 0xFFFFFFFF
                    g, b = divmod(k, 16)
                    buf[i * 4 * Kp + g * 64 + t * 16 + b] = dig
        assert np.array_equal(digit_layout_unpack(buf, rows, K), x)
        assert digit_layout_pad_is_zero(buf, rows, K)
