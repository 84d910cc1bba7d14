"""Pins for the oracle's fixed-point quantisation (CPU only)."""
import numpy as np

from oracle.quant import dequantize, max_qx, quantize_rows


def test_codes_in_window_and_error_half_step():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((16, 300)).astype(np.float32) * 3
    x[3] = 0
    q, s = quantize_rows(x, 127)
    assert q.min() >= -127 and q.max() <= 127
    nz = np.any(x != 0, axis=1)
    assert np.all(np.max(np.abs(q[nz]), axis=1) == 127)
    assert np.all(q[3] == 0) and s[3] == 1.0
    err = np.abs(x.astype(np.float64) - q * s[:, None].astype(np.float64))
    assert np.all(err <= 0.5 * s[:, None] * (1 + 1e-5))


def test_ties_to_even():
    x = np.array([[2.5, -2.5, 0.5, 1.5, 4.0]], dtype=np.float32)
    q, s = quantize_rows(x, 4)
    assert s[0] == 1.0
    assert q.tolist() == [[2, -2, 0, 2, 4]]


def test_window_prevents_wrap():
    """Section 5: codes bounded by q_w, q_x (plus the noise bound) keep every
    inner product of length n inside the signed 32-bit ring range."""
    for n in (8192, 28672):
        qw = 127
        qx = max_qx(n, qw, margin=4)
        worst = n * (qw + 4) * (qx + 4)
        assert worst <= 2 ** 31 - 1
        assert n * (qw + 4) * (qx + 5) > 2 ** 31 - 1
    assert max_qx(8192, 127, 4) == 1997 and max_qx(28672, 127, 4) == 567


def test_dequantize_recovers_product():
    rng = np.random.default_rng(1)
    w = rng.standard_normal((8, 64)).astype(np.float32)
    x = rng.standard_normal((6, 64)).astype(np.float32)
    qw, sw = quantize_rows(w, 127)
    qx, sx = quantize_rows(x, 1997)
    y = dequantize(qx.astype(np.int64) @ qw.astype(np.int64).T, sx, sw)
    ref = x.astype(np.float64) @ w.astype(np.float64).T
    assert np.max(np.abs(y - ref)) < 0.05 * np.max(np.abs(ref))
