"""Integrity check of the server's product (Freivalds' test): Appendix
"Computational integrity", Init W step 3 and online step 4 of the Section
4.2 protocol box. Test infrastructure: the plain CPU definition the GPU path
is checked against.

The client draws check vectors a once per weight matrix and stores the
precomputed product c^T = a^T [W'; Mc_d; ...; Mc_1; ...] (input independent).
After a call it accepts the server's outputs only if

    c^T X' == a^T [Y'; Q]      (paper orientation; t x l on both sides)

which holds for honest outputs by associativity ((a^T W') X' = a^T (W' X'))
and costs O((m + n) l t) instead of the O(m n l) of the product.

Readings (each listed in the design notes):
  * the protocol box compares Y^chk X against a^T Y'; the server computes Y' = W' X',
    so the comparison is made on the masked activations X' (otherwise it
    fails for honest outputs whenever U_x != 0);
  * the Q_i the server returns are covered too, with their own vectors (the
    box checks Y' only; an error in Q_i would pass through unmasking);
  * over Z_{2^32} one uniform vector misses an error E != 0 with probability
    2^-(32 - v), v the smallest 2-adic valuation among E's entries (up to 1/2
    for an error in the top bit only), not the 1/|F| of a field; t vectors
    make that at most 2^-t;
  * vectors are uniform over Z_{2^32}: a_W (t x m) from stream 0x80 and a_i
    (t x r_i) for Q_i from stream 0x90 + i, instance = weight id.

Build orientation (tokens x features), as the rest of the oracle's interface:
A' = X'^T (M x K), Y'^T (M x N), Q_i^T (M x r_i); both sides are t x M.
"""
from __future__ import annotations

from typing import Dict, Sequence, Tuple

import numpy as np

from . import sampling as smp
from .ring import ring_add, ring_matmul


def check_vectors(t: int, N: int, ranks: Sequence[int], seed: int, weight_id: int
                  ) -> Tuple[np.ndarray, Dict[int, np.ndarray]]:
    """a_W (t x N) and {level i: a_i (t x r_i)}, uniform over Z_{2^32}."""
    aW = smp.sample_matrix("uniform", t, N, seed, smp.STREAM_CHECK_W, weight_id)
    aQ = {i: smp.sample_matrix("uniform", t, r, seed, smp.STREAM_CHECK_Q + i, weight_id)
          for i, r in enumerate(ranks, start=1)}
    return aW, aQ


def key(aW: np.ndarray, aQ: Dict[int, np.ndarray], W_masked: np.ndarray, Mc: Dict[int, np.ndarray]) -> np.ndarray:
    """c^T = a_W W' + sum_i a_i (M_i ... M_1) (t x K); W' is N x K, Mc[i] is
    r_i x K."""
    c = ring_matmul(aW, W_masked)
    for i, a in aQ.items():
        c = ring_add(c, ring_matmul(a, Mc[i]))
    return c


def sides(cT: np.ndarray, aW: np.ndarray, aQ: Dict[int, np.ndarray], A_masked: np.ndarray,
          Y_masked_t: np.ndarray, Q_t: Dict[int, np.ndarray]) -> Tuple[np.ndarray, np.ndarray]:
    """(lhs, rhs) = (c^T A'^T, a_W Y'^T^T + sum_i a_i Q_i^T^T), both t x M.
    Y_masked_t is M x N (= Y'^T), Q_t[i] is M x r_i (= Q_i^T)."""
    lhs = ring_matmul(cT, A_masked.T)
    rhs = ring_matmul(aW, Y_masked_t.T)
    for i, a in aQ.items():
        rhs = ring_add(rhs, ring_matmul(a, Q_t[i].T))
    return lhs, rhs


def accept(lhs: np.ndarray, rhs: np.ndarray) -> bool:
    return bool(np.array_equal(lhs, rhs))
