"""Seeded random-shape sweeps of the entry points against the oracle: the
ring product and unmasking (Section 4.2, server step and "Unmasking"), the
samplers, the mask pass, row quantisation and the rotation.

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


SAMPLE_DGAUSS = [(0.5, 4), (1.0, 8), (0.0, 4), (3.2, 15), (0.25, 2), (2.0, 1)]   # thresholds pinned on the host


@pytest.mark.parametrize("block", range(3))
def test_sample_random_shapes(block):
    """Every distribution at random shapes, transposed or not, to ring words,
    to digits or to both (Section 4.2 sampling steps; the fixed-weight rows
    of Example 4.1)."""
    from oracle import sampling as smp
    from tests.gpu_util import pad_is_zero, unpack_digits
    rng = np.random.default_rng(0x53414D50 + block)
    for case in range(CASES_PER_BLOCK):
        kind = str(rng.choice(["uniform", "dgauss", "sparse", "weight"]))
        rows, cols = _size(rng, 1, 700), _size(rng, 1, 3000)
        transposed = kind != "weight" and bool(rng.integers(0, 2))
        sigma, bound = SAMPLE_DGAUSS[int(rng.integers(0, len(SAMPLE_DGAUSS)))]
        lg = int(rng.integers(0, 9))
        t = _size(rng, 1, min(cols, 2048)) if kind == "weight" else 0
        outputs = int(rng.integers(1, 4))       # 1 words, 2 digits, 3 both
        seed, stream, inst = int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 32)), int(rng.integers(0, 2 ** 32))
        print(f"sample case {block}.{case}: {kind} {rows}x{cols} T={transposed} sigma={sigma} bound={bound} "
              f"lg={lg} t={t} outputs={outputs}", flush=True)
        dist = {"uniform": m.DIST_UNIFORM, "dgauss": m.DIST_DGAUSS, "sparse": m.DIST_SPARSE,
                "weight": m.DIST_WEIGHT}[kind]
        r = m.rng(seed, stream, inst, dist, sigma=sigma, bound=bound, log2_inv_density=lg,
                  transposed=transposed, row_weight=t)
        out = torch.full((rows, cols), 99, dtype=torch.int32, device="cuda") if outputs & 1 else None
        dig = Digits.empty(rows, cols) if outputs & 2 else None
        if dig is not None:
            dig.buf.fill_(0x55)
        m.mosaic_sample(r, rows, cols, out=out, out_dig=dig)
        torch.cuda.synchronize()
        kw = dict(sigma=sigma, bound=bound, log2_inv_density=lg, row_weight=t)
        if transposed:
            want = smp.sample_matrix(kind, cols, rows, seed, stream, inst, **kw).T
        else:
            want = smp.sample_matrix(kind, rows, cols, seed, stream, inst, **kw)
        if out is not None:
            assert np.array_equal(to_np_u32(out), want), (block, case)
        if dig is not None:
            assert np.array_equal(unpack_digits(dig), want), (block, case)
            assert pad_is_zero(dig), (block, case)


@pytest.mark.parametrize("block", range(3))
def test_mask_random_shapes(block):
    """X' = X + U + E (Section 4.2, Mask) for int8/16/32 inputs, stored
    transposed or not, with and without U, with no noise or each noise law,
    to ring words, digits or both."""
    from oracle import sampling as smp
    from tests.gpu_util import unpack_digits
    rng = np.random.default_rng(0x4D41534B + block)
    limits = {torch.int8: (np.int8, -128, 128), torch.int16: (np.int16, -32768, 32768),
              torch.int32: (np.int32, -2 ** 31, 2 ** 31)}
    for case in range(CASES_PER_BLOCK):
        rows, cols = _size(rng, 1, 500), _size(rng, 1, 4000)
        dtype = [torch.int8, torch.int16, torch.int32][int(rng.integers(0, 3))]
        transposed = bool(rng.integers(0, 2))
        with_u = bool(rng.integers(0, 2))
        kind = str(rng.choice(["none", "uniform", "dgauss", "sparse"]))
        outputs = int(rng.integers(1, 4))
        print(f"mask case {block}.{case}: {rows}x{cols} {dtype} T={transposed} u={with_u} noise={kind} "
              f"outputs={outputs}", flush=True)
        npdt, lo, hi = limits[dtype]
        x = rng.integers(lo, hi, (cols, rows) if transposed else (rows, cols)).astype(npdt)
        u = _ring(rng, (rows, cols + 3))
        seed, inst = int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 32))
        noise = None if kind == "none" else m.rng(
            seed, 0x51, inst, {"uniform": m.DIST_UNIFORM, "dgauss": m.DIST_DGAUSS, "sparse": m.DIST_SPARSE}[kind],
            sigma=0.5, bound=4, log2_inv_density=3)
        out = torch.full((rows, cols), 99, dtype=torch.int32, device="cuda") if outputs & 1 else None
        dig = Digits.empty(rows, cols) if outputs & 2 else None
        m.mosaic_mask(torch.from_numpy(x).cuda(), to_dev_ring(u)[:, :cols] if with_u else None, noise, rows, cols,
                      out=out, out_dig=dig, x_transposed=transposed)
        torch.cuda.synchronize()
        xv = (x.T if transposed else x).astype(np.int64) & 0xFFFFFFFF
        want = xv + (u[:, :cols].astype(np.int64) if with_u else 0)
        if kind != "none":
            want = want + smp.sample_matrix(kind, rows, cols, seed, 0x51, inst, sigma=0.5, bound=4,
                                            log2_inv_density=3).astype(np.int64)
        want = (want & 0xFFFFFFFF).astype(np.uint32)
        if out is not None:
            assert np.array_equal(to_np_u32(out), want), (block, case)
        if dig is not None:
            assert np.array_equal(unpack_digits(dig), want), (block, case)


@pytest.mark.parametrize("block", range(2))
def test_quantize_random_shapes(block):
    """Row quantisation (Section 5, Pi_Sec-Linear step 1) at random row
    lengths, code ranges and row offsets: codes, digits and scales equal the
    oracle's bit for bit."""
    from oracle import quant as oquant
    from tests.gpu_util import unpack_digits
    rng = np.random.default_rng(0x51554E54 + block)
    for case in range(CASES_PER_BLOCK):
        rows, n = _size(rng, 1, 8), _size(rng, 1, 70000)
        qmax = _size(rng, 1, 1 << 16)
        offset = int(rng.integers(0, 4))
        print(f"quantize case {block}.{case}: {rows}x{n} qmax={qmax} offset={offset}", flush=True)
        x = (rng.standard_normal((rows, n)) * np.exp(rng.uniform(-20, 20, (rows, 1)))).astype(np.float32)
        if rows > 1 and rng.integers(0, 4) == 0:
            x[rows - 1] = 0.0
        wide = torch.zeros((rows, n + 4), dtype=torch.float32, device="cuda")
        wide[:, offset: offset + n] = torch.from_numpy(x).cuda()
        q = torch.empty((rows, n), dtype=torch.int32, device="cuda")
        dig = Digits.empty(rows, n)
        sc = torch.empty(rows, dtype=torch.float32, device="cuda")
        m.mosaic_quantize_rows(wide[:, offset: offset + n], qmax, q=q, q_dig=dig, scale=sc)
        torch.cuda.synchronize()
        qr, sr = oquant.quantize_rows(x, qmax)
        assert np.array_equal(sc.cpu().numpy(), sr), (block, case)
        assert np.array_equal(q.cpu().numpy(), qr), (block, case)
        assert np.array_equal(unpack_digits(dig), qr.view(np.uint32)), (block, case)


@pytest.mark.parametrize("block", range(2))
def test_hadamard_random_shapes(block):
    """Block-diagonal random Hadamard rotations (Section 5, rotation R = H D)
    at random block sizes 2^4..2^15 and block counts, forward or inverse,
    with or without signs: within 1e-5 of each row's peak."""
    from oracle import hadamard as ohad
    from oracle import sampling as smp
    rng = np.random.default_rng(0x48414441 + block)
    for case in range(CASES_PER_BLOCK):
        b = 1 << int(rng.integers(4, 16))
        nb = _size(rng, 1, max(1, 65536 // b))
        n, rows = b * nb, _size(rng, 1, 6)
        inverse, with_signs = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
        print(f"hadamard case {block}.{case}: rows={rows} n={n} b={b} inverse={inverse} signs={with_signs}",
              flush=True)
        x = rng.standard_normal((rows, n)).astype(np.float32)
        x[0, int(rng.integers(0, n))] *= 50.0
        signs = smp.sample_signs(n, int(rng.integers(0, 2 ** 63)), 1) if with_signs else np.ones(n, np.int8)
        y = torch.empty((rows, n), dtype=torch.float32, device="cuda")
        m.mosaic_hadamard_rotate(torch.from_numpy(x).cuda(), y, block=b,
                                 signs=torch.from_numpy(signs).cuda() if with_signs else None, inverse=inverse)
        torch.cuda.synchronize()
        ref = ohad.rotate(x.astype(np.float64), signs, block=b, inverse=inverse)
        err = np.max(np.abs(y.cpu().numpy().astype(np.float64) - ref), axis=1) / np.max(np.abs(ref), axis=1)
        assert np.all(err <= 1e-5), (block, case, float(err.max()))
