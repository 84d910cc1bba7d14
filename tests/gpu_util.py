"""Helpers for the GPU tests: moving ring matrices between torch and numpy."""
import numpy as np
import torch


def to_np_u32(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint32)


def to_dev_ring(x: np.ndarray) -> torch.Tensor:
    """uint32 numpy matrix -> int32 device tensor holding the same bits."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.uint32).view(np.int32)).cuda()


def digits_np(d) -> np.ndarray:
    """Raw bytes of a Digits view's buffer (whole rows)."""
    return d.buf.detach().cpu().numpy()


def unpack_digits(d, rows=None):
    """Ring matrix held by a Digits view (columns col0 .. col0+cols)."""
    from oracle.ring import digit_layout_unpack, padded_k
    raw = digits_np(d)
    r = raw.shape[0] if rows is None else rows
    sub = raw[:r, 4 * d.col0: 4 * d.col0 + 4 * padded_k(d.cols)]
    return digit_layout_unpack(np.ascontiguousarray(sub), r, d.cols)


def pad_is_zero(d) -> bool:
    from oracle.ring import digit_layout_pad_is_zero, padded_k
    raw = digits_np(d)
    sub = raw[:, 4 * d.col0: 4 * d.col0 + 4 * padded_k(d.cols)]
    return digit_layout_pad_is_zero(np.ascontiguousarray(sub), raw.shape[0], d.cols)


def noisy_identity(A, W, params, seed, weight_id, call_id):
    """(A + E_a)(W + E_w)^T mod 2^32 as uint32 (M x N) -- what unmasking must
    return for every mask draw (Section 4.1, eq. approx-error; Section 4.2,
    "Unmasking") -- with E_a, E_w drawn by the oracle's sampler (E_a in the
    build's row-major order of the activations, instance = call id; E_w with
    instance = weight id). float64 products are exact here: every entry of
    the product is below 2^53 in magnitude."""
    from oracle import sampling as smp
    from oracle.ring import lift
    nz = params.noise
    M, K = A.shape
    N = W.shape[0]
    a = A.astype(np.float64)
    b = W.astype(np.float64)
    if nz.kind != "zero":
        a += lift(smp.sample_matrix("dgauss", M, K, seed, smp.STREAM_EX, call_id,
                                    sigma=nz.sigma, bound=nz.bound))
        b += lift(smp.sample_matrix("dgauss", N, K, seed, smp.STREAM_EW, weight_id,
                                    sigma=nz.sigma, bound=nz.bound))
    y = a @ b.T
    del a, b
    return (y.astype(np.int64) & 0xFFFFFFFF).astype(np.uint32)


def code_validity(codes_gpu, scales_gpu, x64, signs, block, qmax, tol=0.02):
    """Checks GPU codes of rows x64 (float64, unrotated) against the oracle's
    float64 rotation and quantisation: scales within 1e-5, codes equal
    wherever x / s is farther than ``tol`` from a rounding tie (the fp32 and
    float64 rotations then round alike), one of the two neighbours
    otherwise. Returns the fraction of ambiguous entries."""
    from oracle import hadamard as ohad
    xr = ohad.rotate(x64, signs, block)
    amax = np.max(np.abs(xr), axis=1)
    s64 = amax / qmax
    assert np.all(np.abs(scales_gpu.astype(np.float64) - s64) <= 1e-5 * s64)
    v = xr / s64[:, None]
    ref = np.rint(v)
    frac = np.abs(v - np.floor(v) - 0.5)
    clear = frac > tol
    got = codes_gpu.astype(np.int64)
    assert np.array_equal(got[clear], ref[clear].astype(np.int64))
    amb = ~clear
    assert np.all((got[amb] == np.floor(v[amb])) | (got[amb] == np.ceil(v[amb])))
    assert np.max(np.abs(got)) <= qmax
    return float(np.mean(amb))
