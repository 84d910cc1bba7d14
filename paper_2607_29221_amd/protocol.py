"""Pi_Sec-Approx-MatMul on one GPU (Section 4.2 protocol box), sequenced from
the C ABI. This module only allocates device buffers and orders the calls;
every arithmetic step is a libmosaic kernel.

Orientation (row-major layout): activations A are M x K (tokens x features),
weights W are N x K (out x in), outputs are M x N. In the paper's notation
A = X^T and the output is (W X)^T; every product below is the transpose of
the protocol box's product and is computed as C = A B^T by mosaic_masked_matmul.

Factors of different levels are concatenated along the inner dimension, in
the slot order (level d, level 1, ..., level d-1):
    Lcat  = [L | S_2 | ... | S_d]                       N x R   (client)
    Jcat  = [J_d | J_1 | ... | J_{d-1}]                 N x R   (client)
    Nccat = [N_1..N_d | N_1 | ... | N_1..N_{d-1}]       K x R   (client)
    rho   = [R^T | T_2^T | ... | T_d^T]                 M x R   (client, per call)
    Bext  = [W' ; M_d..M_1 ; M_1 ; ... ; M_{d-1}..M_1]  (N + R) x K (server)
so that U_a = rho Nccat^T, K_c = rho Jcat^T, [Y' | Q] = A' Bext^T and the
unmask term is Q Lcat^T, exactly the sums of the protocol box.

Random matrices come from Philox streams keyed by the seed: weight-side
material uses the weight id as the counter's instance word, per-call
material the call id.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import torch

from . import mosaic as m
from .mosaic import Digits, padded_k

# stream identifiers (counter word 2), one per random matrix of the protocol
STREAM_EW = 0x10
STREAM_L = 0x11
STREAM_M = 0x20     # + i
STREAM_N = 0x30     # + i
STREAM_S = 0x40     # + i
STREAM_EX = 0x50
STREAM_R = 0x51
STREAM_T = 0x60     # + i
STREAM_SIGNS = 0x70
STREAM_CHECK_W = 0x80   # integrity check vectors for the Y' columns
STREAM_CHECK_Q = 0x90   # + i: integrity check vectors for the Q_i columns


def _noise_rng(params, seed: int, stream: int, instance: int):
    nz = params.noise
    if nz.kind == "zero":
        return None
    if nz.kind != "dgauss":
        raise ValueError(f"unsupported noise kind {nz.kind!r}")
    return m.rng(seed, stream, instance, m.DIST_DGAUSS, sigma=nz.sigma, bound=nz.bound)


def _lpn_rng(params, level: int, seed: int, stream: int, instance: int):
    """Stream of the sparse LPN matrix of ``level`` (S_level, or T_level^T):
    fixed row weight t_level when the parameters give one (Example 4.1),
    else noise rate 2^-s."""
    weights = tuple(getattr(params, "lpn_weights", ()) or ())
    if weights:
        return m.rng(seed, stream, instance, m.DIST_WEIGHT, row_weight=int(weights[level - 2]))
    return m.rng(seed, stream, instance, m.DIST_SPARSE, log2_inv_density=params.sparse_log2_inv_density)


# Token counts up to which a call with both LPN forms available uses the
# sparse gathers: their bytes grow with the token count and reach those of
# the dense slot products at about 64 tokens (measured: sparse 6-19% faster
# at 1 and 8 tokens, 12-30% slower at 64).
SPARSE_LPN_MAX_TOKENS = 16


def _ring_empty(rows: int, cols: int, device) -> torch.Tensor:
    return torch.empty((rows, cols), dtype=torch.int32, device=device)


class MaskedWeight:
    """Init W of the protocol box for one plaintext weight matrix W (N x K,
    int8/int16/int32 on the GPU). Holds the server's Bext and the client's
    unmasking material.

    With ``check_vectors`` = t > 0 it also prepares the integrity check of
    the server's outputs (Freivalds' test; box Init W step 3): check vectors
    a_W (t x N, uniform) for the Y' columns and a_i (t x r_i) for each Q_i,
    and the key c^T = a_W W' + sum_i a_i (M_i ... M_1) (t x K), all held in
    digit layout by the client. One vector misses an error in the top bit
    with probability 1/2 over Z_{2^32}; t vectors bound that by 2^-t.

    At depth >= 2 the LPN matrices can also stay sparse on the client:
    S_{i+1} is kept in compressed rows and multiplied by gathering (S_{i+1}
    Q_i at unmasking), T_{i+1} is drawn inside the gathers into U_a and K_c,
    so their cost per output follows the nonzero count instead of r_i; the
    dense products then run over the level-d slot only. ``sparse_lpn`` None
    (the default) keeps both forms and picks per call from the token count
    (sparse up to SPARSE_LPN_MAX_TOKENS), True keeps only the sparse form,
    False only the dense one. Results are identical either way."""

    def __init__(self, W: torch.Tensor, params, seed: int, weight_id: int = 0, check_vectors: int = 0,
                 sparse_lpn: Optional[bool] = None):
        dev = W.device
        N, K = W.shape
        r = list(params.ranks)
        d = len(r)
        self.params, self.seed, self.weight_id = params, seed, weight_id
        self.N, self.K, self.d = N, K, d
        self.slot_levels = [d] + list(range(1, d))            # level of each slot
        self.slot_ranks = [r[lv - 1] for lv in self.slot_levels]
        self.R = sum(padded_k(c) for c in self.slot_ranks)    # padded inner width
        self.sparse_mode = sparse_lpn
        self.keep_sparse = d >= 2 and sparse_lpn is not False  # compressed S, D_i
        self.keep_dense = not (d >= 2 and sparse_lpn is True)  # every slot in Lcat / Bx
        self.sparse = self.keep_sparse and not self.keep_dense  # sparse-only weight
        self.Rd = padded_k(r[d - 1])                          # width of the sparse calls' products
        U = m.DIST_UNIFORM
        s = seed

        Kp = padded_k(K)
        slot_of = {lv: k for k, lv in enumerate(self.slot_levels)}
        # destinations: the server's Bext rows, and the client's concatenated
        # factors (one buffer each, slots side by side)
        self.Bext = Digits(torch.zeros((N + self.R, 4 * Kp), dtype=torch.int8, device=dev), K)
        self.q_cols, row = [], N
        for ri in self.slot_ranks:
            self.q_cols.append(row)          # column of this slot's Q in [Y' | Q]
            row += padded_k(ri)
        self.n_out = N + self.R
        McTcat = Digits.concat(K, self.slot_ranks, dev)
        bx = torch.empty((K + N, 4 * max(self.R, 64)), dtype=torch.int8, device=dev)
        self.Bx = Digits(bx, self.R)         # [Nccat ; Jcat], the per-call product's operand
        slot_col = [sum(padded_k(c) for c in self.slot_ranks[:k]) for k in range(d)]

        def mc_dst(i):    # M_i ... M_1 (r_i x K): rows of Bext
            r0 = self.q_cols[slot_of[i]]
            return Digits(self.Bext.buf[r0: r0 + r[i - 1]], K)

        def mct_dst(i):   # (M_i ... M_1)^T (K x r_i)
            return McTcat[slot_of[i]]

        def nc_dst(i):    # N_1 ... N_i (K x r_i): upper rows of Bx
            return Digits(bx[:K], r[i - 1], slot_col[slot_of[i]])

        # sparse mode: ring words of M_i..M_1 (r_i x K, partner of S_{i+1} in U_w)
        # and D_i = [(N_1..N_i)^T | J_i^T] (r_i x (K + N), partner of T_{i+1})
        # for the levels i < d that meet a sparse matrix
        self.D: dict = {}
        Mc32: dict = {}
        if self.keep_sparse:
            for i in range(1, d):
                self.D[i] = _ring_empty(r[i - 1], K + N, dev)
                if not self.keep_dense:                       # U_w then needs S_{i+1} Mc_i by gathering
                    Mc32[i] = _ring_empty(r[i - 1], K, dev)

        NcT: List[Digits] = []                # (N_1 ... N_i)^T (r_i x K)
        for i in range(1, d + 1):
            ri = r[i - 1]
            nct = Digits.empty(ri, K, dev)
            keep = i in Mc32
            keep_d = i in self.D
            if i == 1:
                m.mosaic_sample(m.rng(s, STREAM_M + 1, weight_id, U), ri, K, out_dig=mc_dst(1),
                                out=Mc32[1] if keep else None)
                m.mosaic_sample(m.rng(s, STREAM_M + 1, weight_id, U, transposed=True), K, ri, out_dig=mct_dst(1))
                m.mosaic_sample(m.rng(s, STREAM_N + 1, weight_id, U), K, ri, out_dig=nc_dst(1))
                m.mosaic_sample(m.rng(s, STREAM_N + 1, weight_id, U, transposed=True), ri, K, out_dig=nct,
                                out=self.D[1][:, :K] if keep_d else None)
            else:
                rp = r[i - 2]
                Mi = Digits.empty(ri, rp, dev)                  # M_i (r_i x r_{i-1})
                NiT = Digits.empty(ri, rp, dev)                 # N_i^T
                m.mosaic_sample(m.rng(s, STREAM_M + i, weight_id, U), ri, rp, out_dig=Mi)
                m.mosaic_sample(m.rng(s, STREAM_N + i, weight_id, U, transposed=True), ri, rp, out_dig=NiT)
                self._product_to_digits(Mi, mct_dst(i - 1), ri, K, rp, mc_dst(i),
                                        Mc32[i] if keep else None)                      # M_i Mc_{i-1}
                self._product_to_digits(mct_dst(i - 1), Mi, K, ri, rp, mct_dst(i))   # McT_{i-1} M_i^T
                self._product_to_digits(nc_dst(i - 1), NiT, K, ri, rp, nc_dst(i))    # Nc_{i-1} N_i
                self._product_to_digits(NiT, nc_dst(i - 1), ri, K, rp, nct,
                                        self.D[i][:, :K] if keep_d else None)          # N_i^T Nc_{i-1}^T
            NcT.append(nct)

        # client: Lcat = [L | S_2 | ... | S_d] (sparse-only: L alone), and
        # S_{i+1} as compressed rows when the sparse form is kept
        self.Lcat = Digits.concat(N, self.slot_ranks if self.keep_dense else self.slot_ranks[:1], dev)
        m.mosaic_sample(m.rng(s, STREAM_L, weight_id, U), N, r[d - 1], out_dig=self.Lcat[0])
        self.S: dict = {}
        for slot, lv in enumerate(self.slot_levels[1:], start=1):
            srng = _lpn_rng(params, lv + 1, s, STREAM_S + lv + 1, weight_id)
            if self.keep_sparse:
                self.S[lv] = m.mosaic_sparse_csr(srng, N, r[lv - 1], exact=True, device=dev)
            if self.keep_dense:
                m.mosaic_sample(srng, N, r[lv - 1], out_dig=self.Lcat[slot])

        # integrity check vectors (slots of a_Q in the order of Q's columns)
        self.t = int(check_vectors)
        if self.t > 0:
            t = self.t
            if N % 64 == 0:
                # [a_W | a_Q] in one buffer whose columns line up with [Y' | Q]
                cat = Digits.concat(t, [N] + self.slot_ranks, dev)
                self.aW, self.aQ = cat[0], cat[1:]
                self.aWQ: Optional[Digits] = Digits(cat[0].buf, N + self.R, 0)
                self.aQ_all = Digits(cat[0].buf, self.R, N)
            else:
                self.aW = Digits.empty(t, N, dev)
                self.aQ = Digits.concat(t, self.slot_ranks, dev)
                self.aWQ = None
                self.aQ_all = self.aQ[0].whole(self.R)
            m.mosaic_sample(m.rng(s, STREAM_CHECK_W, weight_id, U), t, N, out_dig=self.aW)
            for slot, lv in enumerate(self.slot_levels):
                m.mosaic_sample(m.rng(s, STREAM_CHECK_Q + lv, weight_id, U), t, r[lv - 1], out_dig=self.aQ[slot])
            key_q = _ring_empty(t, K, dev)          # sum_i a_i Mc_i = aQcat McTcat^T
            m.mosaic_masked_matmul(self.aQ_all, McTcat[0].whole(self.R), t, K, self.R, key_q)

        # U_w = Lcat McTcat^T (= L Mc_d + sum S_{i+1} Mc_i); W' = W + U_w + E_w
        U_w = _ring_empty(N, K, dev)
        if self.keep_dense:
            m.mosaic_masked_matmul(self.Lcat[0].whole(self.R), McTcat[0].whole(self.R), N, K, self.R, U_w)
        else:
            m.mosaic_masked_matmul(self.Lcat[0].whole(self.Rd), McTcat[0].whole(self.Rd), N, K, self.Rd, U_w)
            for lv, S in self.S.items():
                m.mosaic_sparse_gather_rows(S, Mc32[lv], K, U_w)
        del McTcat, Mc32
        ew = _noise_rng(params, s, STREAM_EW, weight_id)
        Wm = _ring_empty(N, K, dev) if self.t > 0 else None
        m.mosaic_mask(W, U_w, ew, N, K, out=Wm, out_dig=Digits(self.Bext.buf[:N], K))
        del U_w
        if self.t > 0:
            # key: c^T = a_W W' + key_q, with W'^T in digit layout for the product
            WmT = Digits.empty(K, N, dev)
            m.mosaic_mask(Wm, None, None, K, N, out_dig=WmT, x_transposed=True)
            del Wm
            key_w = _ring_empty(self.t, K, dev)
            m.mosaic_masked_matmul(self.aW, WmT, self.t, K, N, key_w)
            del WmT
            self.cT = Digits.empty(self.t, K, dev)
            m.mosaic_mask(key_w, key_q, None, self.t, K, out_dig=self.cT)
            del key_w, key_q

        # client: J_i = (W + E_w) Nc_i, stored in the lower rows of Bx
        WE = Digits.empty(N, K, dev)
        m.mosaic_mask(W, None, ew, N, K, out_dig=WE)
        for lv in range(1, d + 1):
            ri = r[lv - 1]
            J = _ring_empty(N, ri, dev)
            m.mosaic_masked_matmul(WE, NcT[lv - 1], N, ri, K, J)
            m.mosaic_mask(None, J, None, N, ri, out_dig=Digits(bx[K:], ri, slot_col[slot_of[lv]]))
            if lv in self.D:                                  # J_i^T next to (N_1..N_i)^T
                m.mosaic_masked_matmul(NcT[lv - 1], WE, ri, N, K, self.D[lv][:, K:])
        del WE, NcT
        self.Bx_dense = Digits(bx, r[d - 1])     # the level-d slot (sparse calls)

    def sparse_call(self, M: int) -> bool:
        """Whether a call with M tokens uses the sparse LPN form."""
        if not self.keep_sparse:
            return False
        if not self.keep_dense:
            return True
        return M <= SPARSE_LPN_MAX_TOKENS

    @staticmethod
    def _product_to_digits(a: Digits, b: Digits, rows: int, cols: int, inner: int, out: Digits,
                           words: Optional[torch.Tensor] = None) -> None:
        """out = digits of a b^T; ``words`` (optional) receives the ring words."""
        tmp = _ring_empty(rows, cols, a.buf.device) if words is None else words
        m.mosaic_masked_matmul(a, b, rows, cols, inner, tmp)
        m.mosaic_mask(None, tmp, None, rows, cols, out_dig=out)


@dataclass
class CallBuffers:
    rho: List[Digits]          # [R^T | T_2^T | ...] slots, M x R
    UK: torch.Tensor           # [U_a | K_c], M x (K + N)
    A_masked: Digits           # A' (M x K digits)
    YQ: torch.Tensor           # [Y' | Q], M x (N + R)
    Qdig: List[Digits]         # Q slots in digit layout, M x R
    Y: torch.Tensor            # unmasked output, M x N int32
    check: Optional[tuple] = None   # (lhs, rhs) of the last integrity check formed side by side
    check_diff: Optional[torch.Tensor] = None   # lhs - rhs of the last check in one call


def alloc_call(w: MaskedWeight, M: int, device="cuda") -> CallBuffers:
    return CallBuffers(
        rho=Digits.concat(M, w.slot_ranks, device),
        UK=_ring_empty(M, w.K + w.N, device),
        A_masked=Digits.empty(M, w.K, device),
        YQ=_ring_empty(M, w.n_out, device),
        Qdig=Digits.concat(M, w.slot_ranks, device),
        Y=_ring_empty(M, w.N, device),
    )


def init_x(w: MaskedWeight, M: int, call_id: int, buf: CallBuffers) -> None:
    """Init X (box, online step 1): sample R and T_i, then U_a and K_c in one
    product (E_x is drawn later, inside the mask pass)."""
    p, s, r = w.params, w.seed, list(w.params.ranks)
    m.mosaic_sample(m.rng(s, STREAM_R, call_id, m.DIST_UNIFORM), M, r[w.d - 1], out_dig=buf.rho[0])
    if not w.sparse_call(M):
        for slot, lv in enumerate(w.slot_levels[1:], start=1):
            m.mosaic_sample(_lpn_rng(p, lv + 1, s, STREAM_T + lv + 1, call_id), M, r[lv - 1], out_dig=buf.rho[slot])
        m.mosaic_masked_matmul(buf.rho[0].whole(w.R), w.Bx, M, w.K + w.N, w.R, buf.UK)
        return
    # sparse mode: the level-d slot as a product, then each T_{i+1}^T (M x r_i,
    # a few nonzeros per token, drawn inside the gather) against
    # D_i = [(N_1..N_i)^T | J_i^T]
    m.mosaic_masked_matmul(buf.rho[0].whole(w.Rd), w.Bx_dense.whole(w.Rd), M, w.K + w.N, w.Rd, buf.UK)
    for lv, D in w.D.items():
        m.mosaic_sparse_stream_gather_rows(_lpn_rng(p, lv + 1, s, STREAM_T + lv + 1, call_id),
                                           M, r[lv - 1], D, w.K + w.N, buf.UK)


def mask(w: MaskedWeight, A: torch.Tensor, call_id: int, buf: CallBuffers) -> None:
    """Online step 2: A' = A + U_a + E_a, written in digit layout."""
    M = A.shape[0]
    ex = _noise_rng(w.params, w.seed, STREAM_EX, call_id)
    m.mosaic_mask(A, buf.UK[:, : w.K], ex, M, w.K, out_dig=buf.A_masked)


def server(w: MaskedWeight, M: int, buf: CallBuffers) -> None:
    """Online step 3 on the untrusted side: [Y' | Q] = A' Bext^T."""
    m.mosaic_masked_matmul(buf.A_masked, w.Bext, M, w.n_out, w.K, buf.YQ)


def unmask(w: MaskedWeight, M: int, buf: CallBuffers, y_f32: Optional[torch.Tensor] = None,
           s_rows: Optional[torch.Tensor] = None, s_cols: Optional[torch.Tensor] = None,
           bias: Optional[torch.Tensor] = None) -> None:
    """Online step 5: Y = Y' - K_c - Q Lcat^T (with at most 16 tokens the
    product forms Q's digits from its ring words, else a pass converts Q
    first). In sparse mode the product covers the level-d slot (L Q_d) and
    each S_{i+1} Q_i is subtracted by gathering from Q_i's ring words."""
    r = list(w.params.ranks)
    sparse = w.sparse_call(M)
    # the slots sit side by side in [Y' | Q] with the padded widths of Lcat
    # (and Qdig), and the padding columns of Q are zero (Bext's padding rows
    # are), so one product covers every slot; sparse mode needs slot 0 only
    qw = w.Rd if sparse else w.R
    q_words = buf.YQ[:, w.q_cols[0]: w.q_cols[0] + qw]
    kw = dict(y=buf.Y) if sparse else dict(y=buf.Y, s_rows=s_rows, s_cols=s_cols, y_f32=y_f32, bias=bias)
    if M <= 16 and q_words.data_ptr() % 16 == 0 and q_words.stride(0) % 4 == 0:
        # a few tokens: the product reads Q's ring words as the server wrote
        # them (no conversion pass, one launch fewer per call)
        m.mosaic_unmask_words(buf.YQ[:, : w.N], buf.UK[:, w.K:], q_words, w.Lcat[0].whole(qw), M, w.N, qw, **kw)
    else:
        m.mosaic_mask(None, q_words, None, M, qw, out_dig=buf.Qdig[0].whole(qw))
        m.mosaic_unmask(buf.YQ[:, : w.N], buf.UK[:, w.K:], buf.Qdig[0].whole(qw), w.Lcat[0].whole(qw),
                        M, w.N, qw, **kw)
    if not sparse:
        return
    gathers = [(slot, lv) for slot, lv in enumerate(w.slot_levels) if lv in w.S]
    for k, (slot, lv) in enumerate(gathers):
        c0 = w.q_cols[slot]
        last = k == len(gathers) - 1         # the last gather also writes the dequantised output
        m.mosaic_sparse_gather_cols(w.S[lv], buf.YQ[:, c0: c0 + r[lv - 1]], M, buf.Y, subtract=True,
                                    y_f32=y_f32 if last else None, s_rows=s_rows if last else None,
                                    s_cols=s_cols if last else None, bias=bias if last else None)
    if y_f32 is not None and not gathers:    # dequantise the finished result (no product term)
        m.mosaic_unmask(buf.Y, None, None, None, M, w.N, 0, s_rows=s_rows, s_cols=s_cols, y_f32=y_f32, bias=bias)


def verify(w: MaskedWeight, M: int, buf: CallBuffers, sides: bool = False) -> torch.Tensor:
    """Online step 4 (Freivalds' test) on the server's [Y' | Q]: compares
    lhs = c^T A'^T with rhs = a_W Y'^T + a_Q Q^T (both t x M, on the masked
    activations A' the server multiplied) and returns a one-element int64
    device tensor with the number of entries where they differ: 0 accepts
    the call. Work O((K + N + R) M t), against M K (N + R) for the product.

    When N is a multiple of 64 (a_W and a_Q then sit side by side like Y'
    and Q) and t <= 64, one library call forms d = lhs - rhs, reading
    [Y' | Q] as ring words, and counts its nonzero entries (d is kept in
    buf.check_diff). Otherwise, or with ``sides``, both sides are formed
    and kept in buf.check: rhs from the ring words in two products when N is
    a multiple of 4, else through digit copies of Y' and Q."""
    if w.t <= 0:
        raise ValueError("the weight was prepared without check vectors")
    dev = buf.YQ.device
    t = w.t
    if w.aWQ is not None and t <= 64 and not sides:
        d = _ring_empty(t, M, dev)
        count = torch.empty(1, dtype=torch.int64, device=dev)
        m.mosaic_integrity_check(w.cT, buf.A_masked, w.aWQ, buf.YQ, t, M, w.K, w.N + w.R, d, count)
        buf.check_diff, buf.check = d, None
        return count
    lhs = _ring_empty(t, M, dev)
    m.mosaic_masked_matmul(w.cT, buf.A_masked, t, M, w.K, lhs)
    if w.N % 4 == 0 and t <= 64:
        # straight from the server's ring words (one read of [Y' | Q]; Q's
        # padding columns are zero, as are a_Q's digits there)
        rhs = _ring_empty(t, M, dev)
        m.mosaic_masked_matmul_words(w.aW, buf.YQ[:, : w.N], t, M, w.N, rhs)
        m.mosaic_masked_matmul_words(w.aQ_all, buf.YQ[:, w.N: w.N + w.R], t, M, w.R, rhs, accumulate=True)
        count = torch.empty(1, dtype=torch.int64, device=dev)
        m.mosaic_count_mismatches(lhs, rhs, count)
        buf.check, buf.check_diff = (lhs, rhs), None
        return count
    Ydig = Digits.empty(M, w.N, dev)
    m.mosaic_mask(None, buf.YQ[:, : w.N], None, M, w.N, out_dig=Ydig)
    r = list(w.params.ranks)
    for slot, lv in enumerate(w.slot_levels):
        c0 = w.q_cols[slot]
        m.mosaic_mask(None, buf.YQ[:, c0: c0 + r[lv - 1]], None, M, r[lv - 1], out_dig=buf.Qdig[slot])
    ry = _ring_empty(t, M, dev)
    m.mosaic_masked_matmul(w.aW, Ydig, t, M, w.N, ry)
    rq = _ring_empty(t, M, dev)
    m.mosaic_masked_matmul(w.aQ_all, buf.Qdig[0].whole(w.R), t, M, w.R, rq)
    rhs = _ring_empty(t, M, dev)
    m.mosaic_mask(ry, rq, None, t, M, out=rhs)
    count = torch.empty(1, dtype=torch.int64, device=dev)
    m.mosaic_count_mismatches(lhs, rhs, count)
    buf.check, buf.check_diff = (lhs, rhs), None
    return count


def run_call(w: MaskedWeight, A: torch.Tensor, call_id: int, buf: Optional[CallBuffers] = None) -> CallBuffers:
    M = A.shape[0]
    if buf is None:
        buf = alloc_call(w, M, A.device)
    init_x(w, M, call_id, buf)
    mask(w, A, call_id, buf)
    server(w, M, buf)
    unmask(w, M, buf)
    return buf
