"""Samplers for the mask material of Pi_Sec-Approx-MatMul (Section 4.2 protocol
box), drawn from Philox-4x32-10 streams.

Stream definition (a reading: the paper names no generator). A stream is
identified by (seed, stream_id, instance). Its word t (t >= 0) is word (t mod 4)
of Philox-4x32-10 with

    key     = (seed mod 2^32, seed div 2^32)
    counter = (b mod 2^32, b div 2^32, stream_id, instance),   b = t div 4.

A logical ``rows x cols`` matrix indexes its elements row-major,
e = i * cols + j, and consumes words in that order:

* uniform over Z_{2^32} (the paper's U(Z_{2^k}), Section 4.1): element e is
  word e;
* discrete Gaussian N(Z_{2^k}; 0, sigma^2) (Section 4.1, "Bounded protocol
  error": Pr[k] proportional to exp(-k^2 / (2 sigma^2))), truncated to
  [-B, B]: element e is -B + #{k : word e >= T_k} for the cumulative
  thresholds T_0 <= ... <= T_{2B-1} of ``dgauss_thresholds``;
* sparse LPN noise S(.; mu) (Background, "LWE and LPN": sparse uniform with
  noise rate mu), mu = 2^-s: element e takes words 2e (gate) and 2e+1 (value)
  and is the value word if the top s bits of the gate word are zero, else 0;
* LPN noise of fixed row Hamming weight t (Example 4.1 parameterises the
  LPN levels by t = 80 nonzeros per noise vector): row i of a rows x cols
  matrix consumes words 2 t i .. 2 t i + 2 t - 1. Its t nonzero columns are
  the first t entries of a partial Fisher-Yates shuffle of 0 .. cols-1: step
  j (j = 0 .. t-1) swaps entries j and j + floor(u_j (cols - j) / 2^32) of
  the running permutation, u_j = word 2 t i + 2 j; the entry at the column
  chosen in step j is word 2 t i + 2 j + 1 (a value of 0 is kept as drawn,
  as in the rate-mu sampler). Every t-subset of columns is then chosen with
  probability 1 / C(cols, t) up to the rounding of u_j (cols - j) / 2^32,
  which moves each step's probabilities by less than cols / 2^32;
* random signs d in {+1, -1}^n (Section 5, "Random Hadamard rotation"):
  d_j = +1 if bit 31 of word j is 0, else -1.
"""
from __future__ import annotations

from decimal import Decimal, getcontext
from typing import List

import numpy as np

from . import _cstream
from .philox import philox4x32_np

# Stream identifiers (counter word 2) of every random matrix of the protocol.
# Weight-side material uses instance = weight-matrix id; activation-side
# material uses instance = call id.
STREAM_EW = 0x10          # E_w, full-rank LWE error on the weights
STREAM_L = 0x11           # L, secret left factor (m x r_d)
STREAM_M = 0x20           # + i: M_i, public (r_i x r_{i-1})
STREAM_N = 0x30           # + i: N_i, public (r_{i-1} x r_i)
STREAM_S = 0x40           # + i: S_i, sparse LPN mask (m x r_{i-1})
STREAM_EX = 0x50          # E_x, full-rank LWE error on the activations
STREAM_R = 0x51           # R, secret right factor
STREAM_T = 0x60           # + i: T_i, sparse LPN mask on the activations
STREAM_SIGNS = 0x70       # d, Hadamard rotation signs
STREAM_CHECK_W = 0x80     # integrity check vectors for the Y' outputs (t x m)
STREAM_CHECK_Q = 0x90     # + i: integrity check vectors for the Q_i outputs (t x r_i)


def stream_words(seed: int, stream: int, instance: int, t0: int, count: int) -> np.ndarray:
    """Words t0 .. t0+count-1 of the stream, as uint32 (the C generator of
    oracle/c for long ranges, the numpy one otherwise; the tests check that
    both agree with the scalar definition)."""
    if count <= 0:
        return np.zeros(0, dtype=np.uint32)
    if count >= 4096:
        return _cstream.stream_words(seed, stream, instance, t0, count)
    return stream_words_np(seed, stream, instance, t0, count)


def stream_words_np(seed: int, stream: int, instance: int, t0: int, count: int) -> np.ndarray:
    """stream_words with the vectorised numpy Philox."""
    if count <= 0:
        return np.zeros(0, dtype=np.uint32)
    t = np.arange(t0, t0 + count, dtype=np.uint64)
    b = t >> np.uint64(2)
    lane = (t & np.uint64(3)).astype(np.int64)
    # evaluate each distinct block once
    b_first = int(b[0])
    b_last = int(b[-1])
    blocks = np.arange(b_first, b_last + 1, dtype=np.uint64)
    k0 = seed & 0xFFFFFFFF
    k1 = (seed >> 32) & 0xFFFFFFFF
    out = philox4x32_np(blocks & np.uint64(0xFFFFFFFF), blocks >> np.uint64(32),
                        np.full(blocks.shape, stream, dtype=np.uint64),
                        np.full(blocks.shape, instance, dtype=np.uint64), k0, k1)
    words = np.stack(out, axis=1)           # (n_blocks, 4)
    idx = (b - np.uint64(b_first)).astype(np.int64)
    return words[idx, lane].astype(np.uint32)


def dgauss_thresholds(sigma: float, bound: int) -> List[int]:
    """Cumulative thresholds T_k = floor(2^32 * F_k + 1/2), k = 0 .. 2B-1, where
    F_k = sum_{j=-B}^{-B+k} p_j and p_j = exp(-j^2 / (2 sigma^2)) / Z over the
    support j in [-B, B]. Computed with 60-digit decimal arithmetic."""
    if bound < 0:
        raise ValueError("bound must be >= 0")
    getcontext().prec = 60
    s = Decimal(repr(float(sigma)))
    if s == 0:
        w = [Decimal(1) if j == 0 else Decimal(0) for j in range(-bound, bound + 1)]
    else:
        w = [(-(Decimal(j) ** 2) / (2 * s * s)).exp() for j in range(-bound, bound + 1)]
    z = sum(w)
    out = []
    acc = Decimal(0)
    for k in range(2 * bound):
        acc += w[k]
        out.append(int((acc / z * Decimal(2 ** 32) + Decimal("0.5")).to_integral_value(rounding="ROUND_FLOOR")))
    return out


def _elements(kind: str, e0: int, count: int, seed: int, stream: int, instance: int,
              sigma: float, bound: int, log2_inv_density: int) -> np.ndarray:
    """Elements e0 .. e0+count-1 of a stream matrix (uint32)."""
    if kind == "zero":
        return np.zeros(count, dtype=np.uint32)
    if kind == "uniform":
        return stream_words(seed, stream, instance, e0, count)
    if kind == "dgauss":
        # -B + #{k : T_k <= word}: the count of thresholds at or below the
        # word, which is its right insertion point in the ascending table
        u = stream_words(seed, stream, instance, e0, count).astype(np.uint64)
        th = np.array(dgauss_thresholds(sigma, bound), dtype=np.uint64)
        v = np.searchsorted(th, u, side="right").astype(np.int64) - bound
        return v.astype(np.int32).view(np.uint32)
    if kind == "sparse":
        w = stream_words(seed, stream, instance, 2 * e0, 2 * count)
        gate = w[0::2]
        val = w[1::2]
        s = int(log2_inv_density)
        keep = (gate >> np.uint32(32 - s)) == 0 if s > 0 else np.ones(count, dtype=bool)
        return np.where(keep, val, np.uint32(0)).astype(np.uint32)
    raise ValueError(f"unknown distribution {kind!r}")


def weighted_rows(row_ids, cols: int, t: int, seed: int, stream: int, instance: int):
    """Nonzero columns and values of rows ``row_ids`` of the fixed-weight LPN
    matrix (t nonzeros per row, see the module notes): returns (positions,
    values), two (len(row_ids), t) arrays; positions[:, j] is the column
    chosen in step j of the row's partial shuffle and values[:, j] its
    entry."""
    row_ids = np.asarray(list(row_ids), dtype=np.int64)
    n = row_ids.size
    if not 0 <= t <= cols:
        raise ValueError("row weight must satisfy 0 <= t <= cols")
    if n == 0 or t == 0:
        return np.zeros((n, t), dtype=np.int64), np.zeros((n, t), dtype=np.uint32)
    if np.array_equal(row_ids, np.arange(row_ids[0], row_ids[0] + n)):    # consecutive rows: one range
        words = stream_words(seed, stream, instance, 2 * t * int(row_ids[0]), 2 * t * n).reshape(n, 2 * t)
    else:
        words = np.stack([stream_words(seed, stream, instance, 2 * t * int(i), 2 * t) for i in row_ids])
    u = words[:, 0::2].astype(np.uint64)
    vals = words[:, 1::2].astype(np.uint32)
    perm = np.tile(np.arange(cols, dtype=np.int64), (n, 1))
    rix = np.arange(n)
    for j in range(t):
        k = j + ((u[:, j] * np.uint64(cols - j)) >> np.uint64(32)).astype(np.int64)
        pj = perm[rix, j].copy()
        perm[rix, j] = perm[rix, k]
        perm[rix, k] = pj
    return perm[:, :t].copy(), vals


def sample_weighted(rows: int, cols: int, t: int, seed: int, stream: int, instance: int) -> np.ndarray:
    """The rows x cols fixed-weight LPN matrix as a dense uint32 matrix."""
    out = np.zeros((rows, cols), dtype=np.uint32)
    chunk = 4096
    for r0 in range(0, rows, chunk):
        ids = range(r0, min(rows, r0 + chunk))
        pos, val = weighted_rows(ids, cols, t, seed, stream, instance)
        out[np.arange(r0, r0 + pos.shape[0])[:, None], pos] = val
    return out


def sample_matrix(kind: str, rows: int, cols: int, seed: int, stream: int, instance: int,
                  sigma: float = 0.5, bound: int = 4, log2_inv_density: int = 6,
                  row_weight: int = 0) -> np.ndarray:
    """A logical rows x cols matrix over Z_{2^32} (uint32, two's complement);
    kind "weight" is the fixed-weight LPN matrix with ``row_weight`` nonzeros
    per row."""
    if kind == "weight":
        return sample_weighted(rows, cols, row_weight, seed, stream, instance)
    return _elements(kind, 0, rows * cols, seed, stream, instance, sigma, bound,
                     log2_inv_density).reshape(rows, cols)


def sample_rows(kind: str, row_ids, cols: int, seed: int, stream: int, instance: int,
                sigma: float = 0.5, bound: int = 4, log2_inv_density: int = 6) -> np.ndarray:
    """Rows ``row_ids`` of the logical matrix with ``cols`` columns (any row
    count): row i holds elements i * cols .. i * cols + cols - 1."""
    return np.stack([_elements(kind, int(i) * cols, cols, seed, stream, instance, sigma, bound,
                               log2_inv_density) for i in row_ids])


def sample_signs(n: int, seed: int, instance: int = 0, stream: int = STREAM_SIGNS) -> np.ndarray:
    """d in {+1, -1}^n as int8."""
    w = stream_words(seed, stream, instance, 0, n)
    return np.where((w >> np.uint32(31)) == 0, 1, -1).astype(np.int8)
