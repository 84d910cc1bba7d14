"""Arithmetic over the ring Z_{2^32} (the paper instantiates Z_{2^k} with k = 32,
Section 6.1 "Emulation approach") and the signed-digit form of its elements.

Ring elements are uint32 arrays holding the canonical representative in
[0, 2^32). The product is numpy's uint64 matrix product followed by reduction
mod 2^32: exact, because every 32x32-bit product fits in 64 bits and 2^32
divides 2^64, so wrap-around of the uint64 accumulation does not change the
residue mod 2^32.

Signed digits. The paper emulates one 32-bit multiply-accumulate with 8-bit
multiply-accumulates by splitting each operand into four 8-bit limbs and
recombining with shifts; because only residues mod 2^32 matter, the limb
products a_i * b_j with i + j >= 4 vanish, leaving ten products (Section 6.1).
Here the limbs are balanced: x = sum_{t<4} d_t 256^t (mod 2^32) with every
d_t in [-128, 127]. That representation exists and is unique for every x
(four base-256 digits shifted by -128 cover each residue exactly once).

Digit layout. The GPU path moves ring matrices in a byte layout of these
digits: a rows x K matrix is stored as int8 [rows][Kp/16][4][16] with
Kp = 64 * ceil(K / 64); byte (i, g, t, b) is digit t of element (i, 16 g + b),
and zero for columns >= K. ``digit_layout_unpack`` reads it back.
"""
from __future__ import annotations

import numpy as np

MASK32 = np.uint64(0xFFFFFFFF)


def to_ring(x) -> np.ndarray:
    """Embed integers into Z_{2^32} by their residue (sign extension for
    negative values, Section 5 "embeds W into Z_{2^k}")."""
    return (np.asarray(x).astype(np.int64) & 0xFFFFFFFF).astype(np.uint32)


def lift(x) -> np.ndarray:
    """Centred representative in [-2^31, 2^31) as int32."""
    return np.asarray(x, dtype=np.uint32).view(np.int32)


def ring_add(*xs) -> np.ndarray:
    acc = np.zeros(np.broadcast(*xs).shape, dtype=np.uint64)
    for x in xs:
        acc = acc + np.asarray(x, dtype=np.uint32).astype(np.uint64)
    return (acc & MASK32).astype(np.uint32)


def ring_sub(x, y) -> np.ndarray:
    d = np.asarray(x, dtype=np.uint32).astype(np.uint64) + (np.uint64(1 << 32) -
                                                            np.asarray(y, dtype=np.uint32).astype(np.uint64))
    return (d & MASK32).astype(np.uint32)


def ring_matmul(x, y) -> np.ndarray:
    """x @ y over Z_{2^32}: x (a x b), y (b x c) -> (a x c)."""
    x = np.asarray(x, dtype=np.uint32).astype(np.uint64)
    y = np.asarray(y, dtype=np.uint32).astype(np.uint64)
    return ((x @ y) & MASK32).astype(np.uint32)


def signed_digits(x) -> np.ndarray:
    """Balanced base-256 digits of ring elements: shape (..., 4) int8 with
    x = sum_t d_t 256^t (mod 2^32), d_t in [-128, 127]. Digit t is the centred
    residue of the remaining value mod 256; the remainder is divided by 256."""
    v = np.asarray(x, dtype=np.uint32).astype(np.int64)
    out = np.empty(v.shape + (4,), dtype=np.int8)
    for t in range(4):
        r = v & 0xFF
        d = np.where(r >= 128, r - 256, r)
        out[..., t] = d
        v = ((v - d) >> 8) & 0xFFFFFFFF
    return out


def from_signed_digits(d) -> np.ndarray:
    """Inverse of ``signed_digits``: sum_t d_t 256^t mod 2^32."""
    d = np.asarray(d).astype(np.int64)
    acc = np.zeros(d.shape[:-1], dtype=np.int64)
    for t in range(4):
        acc = acc + d[..., t] * (256 ** t)
    return (acc & 0xFFFFFFFF).astype(np.uint32)


def padded_k(K: int) -> int:
    return 64 * ((K + 63) // 64)


def digit_layout_unpack(buf, rows: int, K: int, row_pitch: int | None = None) -> np.ndarray:
    """Read a rows x K ring matrix from the digit byte layout."""
    Kp = padded_k(K)
    pitch = 4 * Kp if row_pitch is None else row_pitch
    raw = np.frombuffer(np.ascontiguousarray(buf).tobytes(), dtype=np.int8)
    raw = raw[: rows * pitch].reshape(rows, pitch)[:, : 4 * Kp]
    g = raw.reshape(rows, Kp // 16, 4, 16)               # [row][group][digit][byte]
    d = np.transpose(g, (0, 1, 3, 2)).reshape(rows, Kp, 4)  # [row][col][digit]
    return from_signed_digits(d[:, :K, :])


def digit_layout_pad_is_zero(buf, rows: int, K: int) -> bool:
    """True if every digit byte of the padding columns K .. Kp-1 is zero."""
    Kp = padded_k(K)
    raw = np.frombuffer(np.ascontiguousarray(buf).tobytes(), dtype=np.int8)[: rows * 4 * Kp]
    g = raw.reshape(rows, Kp // 16, 4, 16)
    d = np.transpose(g, (0, 1, 3, 2)).reshape(rows, Kp, 4)
    return bool(np.all(d[:, K:, :] == 0))
