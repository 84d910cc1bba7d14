"""Philox counter-based generator (Salmon, Moraes, Dror, Shaw, "Parallel random
numbers: as easy as 1, 2, 3", SC'11), restated from that paper.

The MOSAIC paper does not name a generator for its mask material; both the
oracle and the GPU kernels draw it from Philox-4x32 with 10 rounds.

Philox-4xW: the state is four W-bit words (c0, c1, c2, c3) (the counter) and a
key of two W-bit words (k0, k1). One round multiplies c0 and c2 by fixed odd
constants, producing double-width products (hi, lo), and outputs

    (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0)).

Between rounds the key is advanced by a Weyl sequence (k0 += W0, k1 += W1,
mod 2^W); round j (0-based) uses key + j*(W0, W1).

Constants (from the SC'11 paper): for W = 32 the multipliers are 0xD2511F53 and
0xCD9E8D57; for W = 64, 0xD2E7470EE14C6C93 and 0xCA5A826395121157. The Weyl
increments are the fractional parts of the golden ratio and of sqrt(3) scaled
to W bits (the tests recompute them from those closed forms).

``philox_generic`` is the scalar reference for any W; ``philox4x32_np`` is the
same function for W = 32 vectorised over numpy arrays. The tests pin the
generic function's W = 64 instance against ``numpy.random.Philox`` (a
Philox-4x64-10 implementation), its W = 32 instance and the vectorised one
against rocRAND's Philox4x32-10 block function (built on the host from
rocRAND's open-source header), and the vectorised one against the generic one.
"""
from __future__ import annotations

from typing import Sequence, Tuple

import numpy as np

PHILOX_CONSTANTS = {
    32: dict(M=(0xD2511F53, 0xCD9E8D57), W=(0x9E3779B9, 0xBB67AE85)),
    64: dict(M=(0xD2E7470EE14C6C93, 0xCA5A826395121157),
             W=(0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)),
}


def philox_generic(ctr: Sequence[int], key: Sequence[int], width: int = 32,
                   rounds: int = 10) -> Tuple[int, int, int, int]:
    """Philox-4x``width`` with ``rounds`` rounds on Python integers."""
    mask = (1 << width) - 1
    m0, m1 = PHILOX_CONSTANTS[width]["M"]
    w0, w1 = PHILOX_CONSTANTS[width]["W"]
    c0, c1, c2, c3 = (int(v) & mask for v in ctr)
    k0, k1 = (int(v) & mask for v in key)
    for _ in range(rounds):
        p0 = m0 * c0
        p1 = m1 * c2
        hi0, lo0 = p0 >> width, p0 & mask
        hi1, lo1 = p1 >> width, p1 & mask
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
        k0 = (k0 + w0) & mask
        k1 = (k1 + w1) & mask
    return c0, c1, c2, c3


def philox4x32_np(c0, c1, c2, c3, k0: int, k1: int, rounds: int = 10):
    """Vectorised Philox-4x32: counters are uint64 arrays holding 32-bit values
    (products of two 32-bit values fit exactly in uint64)."""
    m32 = np.uint64(0xFFFFFFFF)
    sh = np.uint64(32)
    m0, m1 = (np.uint64(v) for v in PHILOX_CONSTANTS[32]["M"])
    w0, w1 = PHILOX_CONSTANTS[32]["W"]
    c0 = np.asarray(c0, dtype=np.uint64) & m32
    c1 = np.asarray(c1, dtype=np.uint64) & m32
    c2 = np.asarray(c2, dtype=np.uint64) & m32
    c3 = np.asarray(c3, dtype=np.uint64) & m32
    k0 = int(k0) & 0xFFFFFFFF
    k1 = int(k1) & 0xFFFFFFFF
    for _ in range(rounds):
        p0 = m0 * c0
        p1 = m1 * c2
        hi0, lo0 = p0 >> sh, p0 & m32
        hi1, lo1 = p1 >> sh, p1 & m32
        c0, c1, c2, c3 = hi1 ^ c1 ^ np.uint64(k0), lo1, hi0 ^ c3 ^ np.uint64(k1), lo0
        k0 = (k0 + w0) & 0xFFFFFFFF
        k1 = (k1 + w1) & 0xFFFFFFFF
    return c0, c1, c2, c3
