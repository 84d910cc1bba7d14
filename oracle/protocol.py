"""Pi_Sec-Approx-MatMul (Section 4.2 protocol box; Section 4.1 for depth 1),
written in the paper's orientation and notation over Z_{2^32}.

Paper orientation: W is m x n (weights), X is n x l (activations), Y = W X.
The build's row-major activations are A = X^T (l x n) and its outputs are
Y^T (l x m); ``run`` converts at the boundary only.

Readings where the paper is ambiguous (listed with reasons in the design notes):
* the sparse masks are S_{i+1} in Z^{m x r_i} and T_{i+1} in Z^{r_i x l}, the
  only dimensions under which S_{i+1} (M_i ... M_1) and N_1 ... N_i T_{i+1}
  are defined (the protocol box prints r_i x r_{i-1} and r_{i-1} x r_i);
* the chains M_i ... M_1 and N_1 ... N_i start from M_1 in Z^{r_1 x n} and
  N_1 in Z^{n x r_1} (r_0 = n);
* activation-side random matrices (R, E_x, T_i) are drawn element by element
  in the build's row-major order of their transposes (the order in which the
  GPU visits them); weight-side ones in the paper's orientation.

Init W computes U_w, J_i and W' = W + U_w (box "Init W" steps 1-5; the
Freivalds vector of step 4 is omitted: integrity checking is not part of the
masked product). Init X samples R, E_x, T_i and forms U_x and K (steps 1a-1c).
The server returns Y' = W' X' and Q_i = (M_i ... M_1) X'; unmasking outputs
Y' - K - L Q_d - sum_i S_{i+1} Q_i.

Expanding W' X' shows that this unmasked value equals (W + E_w)(X + E_x)
exactly in the ring, for any mask draw; that is the identity the tests pin.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import sampling as smp
from .ring import ring_add, ring_matmul, ring_sub, to_ring


@dataclass
class WeightState:
    W: np.ndarray                       # m x n plaintext embedded in the ring
    E_w: np.ndarray                     # m x n
    L: np.ndarray                       # m x r_d
    M: List[np.ndarray]                 # M_i, r_i x r_{i-1}
    N: List[np.ndarray]                 # N_i, r_{i-1} x r_i
    S: List[Optional[np.ndarray]]       # S[i] = S_{i+1} (m x r_i) for i = 1..d-1; index 0 unused
    Mc: List[np.ndarray]                # Mc[i-1] = M_i ... M_1 (r_i x n)
    Nc: List[np.ndarray]                # Nc[i-1] = N_1 ... N_i (n x r_i)
    J: List[np.ndarray]                 # J[i-1] = (W + E_w) N_1 ... N_i (m x r_i)
    U_w: np.ndarray                     # m x n
    W_masked: np.ndarray                # W' (m x n)


@dataclass
class CallState:
    R: np.ndarray                       # r_d x l
    E_x: np.ndarray                     # n x l
    T: List[Optional[np.ndarray]]       # T[i] = T_{i+1} (r_i x l); index 0 unused
    U_x: np.ndarray                     # n x l
    K: np.ndarray                       # m x l


def _noise(params, rows, cols, seed, stream, instance, transposed=False):
    nz = params.noise
    if nz.kind == "zero":
        return np.zeros((rows, cols), dtype=np.uint32)
    if transposed:
        return smp.sample_matrix("dgauss", cols, rows, seed, stream, instance,
                                 sigma=nz.sigma, bound=nz.bound).T.copy()
    return smp.sample_matrix("dgauss", rows, cols, seed, stream, instance,
                             sigma=nz.sigma, bound=nz.bound)


def _lpn(params, level: int, rows: int, cols: int, seed: int, stream: int, instance: int) -> np.ndarray:
    """The sparse LPN matrix of level ``level`` (S_level or T_level^T, rows x
    cols): fixed row Hamming weight t_level when the parameters give one
    (Example 4.1), else the rate-2^-s sampler."""
    w = tuple(getattr(params, "lpn_weights", ()) or ())
    if w:
        return smp.sample_matrix("weight", rows, cols, seed, stream, instance, row_weight=w[level - 2])
    return smp.sample_matrix("sparse", rows, cols, seed, stream, instance,
                             log2_inv_density=params.sparse_log2_inv_density)


def client_cost_per_row(params) -> int:
    """The client's multiplications per output element of unmasking (and per
    input element of masking), r_d + sum_{i=2}^{d} t_i: the dense level-d
    factor plus one product per nonzero of each sparse level (Section 4.2
    cost analysis, Table "lpn-tradeoff"). Requires fixed row weights for
    d >= 2."""
    r = list(params.ranks)
    w = list(getattr(params, "lpn_weights", ()) or ())
    if len(w) != len(r) - 1:
        raise ValueError("the cost needs a row weight for every LPN level")
    return r[-1] + sum(w)


def init_w(W_plain: np.ndarray, params, seed: int, weight_id: int) -> WeightState:
    """Init W of the protocol box for a plaintext m x n weight matrix."""
    W = to_ring(W_plain)
    m, n = W.shape
    r = list(params.ranks)
    d = len(r)
    dims = [n] + r                                    # r_0 = n
    # step 1: sample L, M_i, N_i, E_w, S_i
    L = smp.sample_matrix("uniform", m, r[d - 1], seed, smp.STREAM_L, weight_id)
    M = [smp.sample_matrix("uniform", dims[i], dims[i - 1], seed, smp.STREAM_M + i, weight_id)
         for i in range(1, d + 1)]
    N = [smp.sample_matrix("uniform", dims[i - 1], dims[i], seed, smp.STREAM_N + i, weight_id)
         for i in range(1, d + 1)]
    E_w = _noise(params, m, n, seed, smp.STREAM_EW, weight_id)
    S: List[Optional[np.ndarray]] = [None] * d
    for i in range(1, d):
        S[i] = _lpn(params, i + 1, m, r[i - 1], seed, smp.STREAM_S + i + 1, weight_id)
    # chains M_i ... M_1 and N_1 ... N_i
    Mc = [M[0]]
    Nc = [N[0]]
    for i in range(2, d + 1):
        Mc.append(ring_matmul(M[i - 1], Mc[-1]))
        Nc.append(ring_matmul(Nc[-1], N[i - 1]))
    # step 2: U_w = L (M_d ... M_1) + sum_{i=1}^{d-1} S_{i+1} (M_i ... M_1) + E_w
    U_w = ring_matmul(L, Mc[d - 1])
    for i in range(1, d):
        U_w = ring_add(U_w, ring_matmul(S[i], Mc[i - 1]))
    U_w = ring_add(U_w, E_w)
    # step 3: J_i = (W + E_w) N_1 ... N_i
    WE = ring_add(W, E_w)
    J = [ring_matmul(WE, Nc[i - 1]) for i in range(1, d + 1)]
    # step 5: W' = W + U_w
    return WeightState(W=W, E_w=E_w, L=L, M=M, N=N, S=S, Mc=Mc, Nc=Nc, J=J,
                       U_w=U_w, W_masked=ring_add(W, U_w))


def init_x(ws: WeightState, l: int, params, seed: int, call_id: int) -> CallState:
    """Init X (box, online step 1): sample R, E_x, T_i; form U_x and K."""
    r = list(params.ranks)
    d = len(r)
    n = ws.W.shape[1]
    # step 1a; activation-side matrices are drawn in row-major order of their transposes
    R = smp.sample_matrix("uniform", l, r[d - 1], seed, smp.STREAM_R, call_id).T.copy()
    E_x = _noise(params, n, l, seed, smp.STREAM_EX, call_id, transposed=True)
    T: List[Optional[np.ndarray]] = [None] * d
    for i in range(1, d):
        T[i] = _lpn(params, i + 1, l, r[i - 1], seed, smp.STREAM_T + i + 1, call_id).T.copy()
    # step 1b: U_x = N_1...N_d R + sum_{i=1}^{d-1} N_1...N_i T_{i+1} + E_x
    U_x = ring_matmul(ws.Nc[d - 1], R)
    for i in range(1, d):
        U_x = ring_add(U_x, ring_matmul(ws.Nc[i - 1], T[i]))
    U_x = ring_add(U_x, E_x)
    # step 1c: K = J_d R + sum_{i=1}^{d-1} J_i T_{i+1}
    K = ring_matmul(ws.J[d - 1], R)
    for i in range(1, d):
        K = ring_add(K, ring_matmul(ws.J[i - 1], T[i]))
    return CallState(R=R, E_x=E_x, T=T, U_x=U_x, K=K)


def mask(X: np.ndarray, cs: CallState) -> np.ndarray:
    """Online step 2: X' = X + U_x."""
    return ring_add(to_ring(X), cs.U_x)


def server(ws: WeightState, X_masked: np.ndarray):
    """Online step 3 (untrusted accelerator): Y' = W' X', Q_i = (M_i...M_1) X'."""
    Y_masked = ring_matmul(ws.W_masked, X_masked)
    Q = [ring_matmul(ws.Mc[i], X_masked) for i in range(len(ws.Mc))]
    return Y_masked, Q


def unmask(ws: WeightState, cs: CallState, Y_masked: np.ndarray, Q: List[np.ndarray]) -> np.ndarray:
    """Online step 5: Y = Y' - K - L Q_d - sum_{i=1}^{d-1} S_{i+1} Q_i."""
    d = len(Q)
    Y = ring_sub(Y_masked, cs.K)
    Y = ring_sub(Y, ring_matmul(ws.L, Q[d - 1]))
    for i in range(1, d):
        Y = ring_sub(Y, ring_matmul(ws.S[i], Q[i - 1]))
    return Y


@dataclass
class RunResult:
    ws: WeightState
    cs: CallState
    X_masked: np.ndarray
    Y_masked: np.ndarray
    Q: List[np.ndarray]
    Y: np.ndarray                        # m x l ring element
    extras: dict = field(default_factory=dict)

    # build-orientation views (row-major, tokens first)
    @property
    def A_masked(self):
        return self.X_masked.T

    @property
    def Y_out(self):
        return self.Y.T


def run(A_plain: np.ndarray, W_plain: np.ndarray, params, seed: int, weight_id: int = 0,
        call_id: int = 0) -> RunResult:
    """Init W, Init X, mask, server product and unmask for A (l x n, build
    orientation) and W (m x n)."""
    ws = init_w(W_plain, params, seed, weight_id)
    X = np.asarray(A_plain).T
    cs = init_x(ws, X.shape[1], params, seed, call_id)
    Xm = mask(X, cs)
    Ym, Q = server(ws, Xm)
    Y = unmask(ws, cs, Ym, Q)
    return RunResult(ws=ws, cs=cs, X_masked=Xm, Y_masked=Ym, Q=Q, Y=Y)


def sampled_depth1(A_rows: np.ndarray, W_rows: np.ndarray, I, J, K: int, params, seed: int,
                   weight_id: int, call_id: int) -> dict:
    """Sampled outputs of the depth-1 protocol (Section 4.1) for token rows I
    (A_rows = A[I], build orientation) and weight rows J (W_rows = W[J]),
    computed from the definitions without forming the full matrices:

        W'[J] = W[J] + E_w[J] + L[J] M          (weight mask)
        X'^T[I] = A[I] + R^T[I] N^T + E_x^T[I]  (activation mask)
        Y'^T[I, J] = X'^T[I] W'[J]^T,  Q^T[I] = X'^T[I] M^T
        J_w[J] = (W[J] + E_w[J]) N,   K^T[I, J] = R^T[I] J_w[J]^T
        Y^T[I, J] = Y'^T[I, J] - K^T[I, J] - Q^T[I] L[J]^T

    M (r x K) and N (K x r) are drawn in full; every other matrix only at
    the sampled rows."""
    r = params.ranks[0]
    nz = params.noise
    kind = "zero" if nz.kind == "zero" else "dgauss"
    M_ = smp.sample_matrix("uniform", r, K, seed, smp.STREAM_M + 1, weight_id)
    N_ = smp.sample_matrix("uniform", K, r, seed, smp.STREAM_N + 1, weight_id)
    L_J = smp.sample_rows("uniform", J, r, seed, smp.STREAM_L, weight_id)
    Ew_J = smp.sample_rows(kind, J, K, seed, smp.STREAM_EW, weight_id, sigma=nz.sigma, bound=nz.bound)
    Rt_I = smp.sample_rows("uniform", I, r, seed, smp.STREAM_R, call_id)
    Ex_I = smp.sample_rows(kind, I, K, seed, smp.STREAM_EX, call_id, sigma=nz.sigma, bound=nz.bound)
    WE = ring_add(to_ring(W_rows), Ew_J)
    Wm = ring_add(WE, ring_matmul(L_J, M_))
    Ua_noE = ring_matmul(Rt_I, N_.T)
    Am = ring_add(to_ring(A_rows), Ua_noE, Ex_I)
    Ym = ring_matmul(Am, Wm.T)
    Q = ring_matmul(Am, M_.T)
    Jw = ring_matmul(WE, N_)
    Kc = ring_matmul(Rt_I, Jw.T)
    Y = ring_sub(ring_sub(Ym, Kc), ring_matmul(Q, L_J.T))
    ident = ring_matmul(ring_add(to_ring(A_rows), Ex_I), WE.T)
    return dict(W_masked=Wm, U_a=Ua_noE, A_masked=Am, Y_masked=Ym, Q=Q, K_c=Kc, Y=Y, identity=ident,
                E_w=Ew_J, E_x=Ex_I)


# ---------------------------------------------------------------------------
# Depth 1 (Section 4.1) in the build's row-major orientation, with the ring
# products of the plain C leg (oracle/c/ring_oracle.c, all host cores): the
# same streams and the same sums as init_w / init_x / mask / server / unmask
# above, for the CPU baseline at workload sizes.
# ---------------------------------------------------------------------------
@dataclass
class Depth1Weight:
    W_masked: np.ndarray    # W' = W + E_w + L M     (N x K)
    M: np.ndarray           # M_1                    (r x K)
    N: np.ndarray           # N_1                    (K x r)
    L: np.ndarray           # L                      (N x r)
    J: np.ndarray           # J_1 = (W + E_w) N_1    (N x r)


def init_w_depth1_c(W_plain: np.ndarray, params, seed: int, weight_id: int) -> Depth1Weight:
    """Init W (box steps 1-5 at d = 1) for W (N x K)."""
    from . import _cring
    N_, K = W_plain.shape
    r = params.ranks[0]
    L = smp.sample_matrix("uniform", N_, r, seed, smp.STREAM_L, weight_id)
    M = smp.sample_matrix("uniform", r, K, seed, smp.STREAM_M + 1, weight_id)
    Nm = smp.sample_matrix("uniform", K, r, seed, smp.STREAM_N + 1, weight_id)
    WE = ring_add(to_ring(W_plain), _noise(params, N_, K, seed, smp.STREAM_EW, weight_id))
    Wm = ring_add(WE, _cring.ring_matmul_nt(L, np.ascontiguousarray(M.T)))
    J = _cring.ring_matmul_nt(WE, np.ascontiguousarray(Nm.T))
    return Depth1Weight(W_masked=Wm, M=M, N=Nm, L=L, J=J)


def call_depth1_c(w: Depth1Weight, A_plain: np.ndarray, params, seed: int, call_id: int) -> dict:
    """Init X, mask, server product and unmasking for A (M x K tokens):
        U_a = R^T N^T,  K_c = R^T J^T,  A' = A + U_a + E_a,
        Y' = A' W'^T,  Q^T = A' M^T,  Y = Y' - K_c - Q^T L^T."""
    from . import _cring
    Mt, K = A_plain.shape
    r = w.M.shape[0]
    Rt = smp.sample_matrix("uniform", Mt, r, seed, smp.STREAM_R, call_id)
    Ea = _noise(params, Mt, K, seed, smp.STREAM_EX, call_id)
    Ua = _cring.ring_matmul_nt(Rt, w.N)
    Kc = _cring.ring_matmul_nt(Rt, w.J)
    Am = ring_add(to_ring(A_plain), Ua, Ea)
    Ym = _cring.ring_matmul_nt(Am, w.W_masked)
    Qt = _cring.ring_matmul_nt(Am, w.M)
    Y = ring_sub(ring_sub(Ym, Kc), _cring.ring_matmul_nt(Qt, w.L))
    return dict(U_a=Ua, K_c=Kc, A_masked=Am, Y_masked=Ym, Q=Qt, Y=Y, E_a=Ea)
