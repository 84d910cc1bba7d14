"""Seeded random-shape sweeps of the ring product and of unmasking against
the oracle's ring arithmetic (Section 4.2, server step and "Unmasking").

The fixed cases elsewhere pin the boundaries of each kernel; these draw row
counts, output widths, inner dimensions and ranks at random across those
boundaries, so that the launch selection (decode kernel up to 64 rows, tiled
kernel with or without split-K beyond, word or digit operands, one-pass or
two-phase unmasking) meets shapes nobody chose by hand. Every output is
compared bit for bit. Each case prints its shape before it runs."""
import numpy as np
import pytest
import torch

from oracle.ring import ring_matmul, ring_sub
from paper_2607_29221_amd import mosaic as m
from paper_2607_29221_amd.mosaic import Digits
from tests.gpu_util import to_dev_ring, to_np_u32

pytestmark = pytest.mark.gpu

CASES_PER_BLOCK = 12


def _ring(rng, shape):
    return rng.integers(0, 2 ** 32, shape, dtype=np.uint64).astype(np.uint32)


def _size(rng, lo, hi):
    """Half the draws log-uniform (small and edge sizes), half uniform (sizes
    spanning many tiles)."""
    if rng.integers(0, 2):
        return int(rng.integers(lo, hi + 1))
    return min(hi, int(np.exp(rng.uniform(np.log(lo), np.log(hi + 1)))))


def _digits(x):
    rows, cols = x.shape
    d = Digits.empty(rows, max(cols, 1))
    if rows and cols:
        m.mosaic_mask(to_dev_ring(x), None, None, rows, cols, out_dig=d)
    return d


def _product_shape(rng):
    """Rows across the decode/tiled boundary, ragged N and K; at most about
    4e8 multiply-adds so the oracle's product stays fast."""
    M = _size(rng, 1, 400)
    N = _size(rng, 1, 3000)
    K = _size(rng, 1, 5000)
    while M * N * K > 4e8:
        K = max(1, K // 2)
    return M, N, K


@pytest.mark.parametrize("block", range(4))
def test_masked_matmul_random_shapes(block):
    rng = np.random.default_rng(0x52414E44 + block)
    for case in range(CASES_PER_BLOCK):
        M, N, K = _product_shape(rng)
        words = M <= 64 and bool(rng.integers(0, 2))
        print(f"product case {block}.{case}: M={M} N={N} K={K} words={words}", flush=True)
        a, b = _ring(rng, (M, K)), _ring(rng, (N, K))
        A = _digits(a)
        C = torch.full((M, N), 7, dtype=torch.int32, device="cuda")
        if words:
            Kw = K + (-K) % 4
            wide = _ring(rng, (N, Kw + 4))
            wide[:, :K] = b
            m.mosaic_masked_matmul_words(A, to_dev_ring(wide)[:, :K], M, N, K, C)
        else:
            m.mosaic_masked_matmul(A, _digits(b), M, N, K, C)
        torch.cuda.synchronize()
        assert np.array_equal(to_np_u32(C), ring_matmul(a, b.T)), (block, case, M, N, K, words)


@pytest.mark.parametrize("block", range(4))
def test_unmask_random_shapes(block):
    """Y = Y' - K_c - Q L^T with or without K_c, written to a separate buffer
    or in place over Y' or K_c; Q as digits for every row count and as ring
    words (at a column offset of a wider buffer) up to 16 rows."""
    rng = np.random.default_rng(0x554E4D53 + block)
    for case in range(CASES_PER_BLOCK):
        M = _size(rng, 1, 300) if rng.integers(0, 4) == 0 else int(rng.integers(1, 65))
        N = _size(rng, 1, 2500)
        R = int(rng.choice([0, 64, 1024, 1536])) if rng.integers(0, 3) == 0 else _size(rng, 1, 1800)
        with_k = bool(rng.integers(0, 2))
        target = str(rng.choice(["new", "ym", "kc"] if with_k else ["new", "ym"]))
        words = M <= 16 and R > 0 and bool(rng.integers(0, 2))
        print(f"unmask case {block}.{case}: M={M} N={N} R={R} with_k={with_k} y={target} words={words}", flush=True)
        ym, kc, q, l = _ring(rng, (M, N)), _ring(rng, (M, N)), _ring(rng, (M, R)), _ring(rng, (N, R))
        want = ring_sub(ym, kc) if with_k else ym.copy()
        if R:
            want = ring_sub(want, ring_matmul(q, l.T))
        ymd = to_dev_ring(ym)
        kcd = to_dev_ring(kc) if with_k else None
        y = {"new": torch.empty((M, N), dtype=torch.int32, device="cuda"), "ym": ymd, "kc": kcd}[target]
        L = _digits(l) if R else None
        if words:
            R4 = R + (-R) % 4
            wide = _ring(rng, (M, R4 + 8))
            wide[:, 4:4 + R] = q
            m.mosaic_unmask_words(ymd, kcd, to_dev_ring(wide)[:, 4:4 + R], L, M, N, R, y=y)
        else:
            m.mosaic_unmask(ymd, kcd, _digits(q) if R else None, L, M, N, R, y=y)
        torch.cuda.synchronize()
        assert np.array_equal(to_np_u32(y), want), (block, case, M, N, R, with_k, target, words)
