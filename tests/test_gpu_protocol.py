"""Pi_Sec-Approx-MatMul on the GPU against the oracle, intermediate by
intermediate, on the single-masked-matmul workload (A 64 x 512, W 512 x 512,
int8 in [-127, 127], seed 0) and on ragged shapes, for depths 1 to 3."""
import numpy as np
import pytest
import torch

from oracle import protocol as oproto
from oracle.ring import lift, ring_add, ring_matmul, ring_sub, to_ring
from paper_2607_29221_amd import protocol as gproto
from synthetic_inputs import (PARAMS_D1_SMALL_R128, PARAMS_D2_SPARSE, PARAMS_D3_SPARSE_SMALL, NoiseSpec,
                              ProtocolParams, SMALL_CASE, int8_operands)
from tests.gpu_util import to_np_u32, unpack_digits

pytestmark = pytest.mark.gpu

SEED = 20260701


def _check_run(A, W, params, seed, weight_id=1, call_id=2):
    ref = oproto.run(A, W, params, seed, weight_id, call_id)
    Wd = torch.from_numpy(W).cuda()
    Ad = torch.from_numpy(A).cuda()
    w = gproto.MaskedWeight(Wd, params, seed, weight_id, sparse_lpn=False)     # dense layout: every factor in Lcat/Bx
    buf = gproto.run_call(w, Ad, call_id)
    torch.cuda.synchronize()
    N, K = W.shape
    M = A.shape[0]
    d = params.depth
    ws, cs = ref.ws, ref.cs

    # Init W: server operand and client material
    from paper_2607_29221_amd.mosaic import Digits
    assert np.array_equal(unpack_digits(Digits(w.Bext.buf[:N], K)), ws.W_masked)
    for slot, lv in enumerate(w.slot_levels):
        r0 = w.q_cols[slot]
        ri = params.ranks[lv - 1]
        assert np.array_equal(unpack_digits(Digits(w.Bext.buf[r0:r0 + ri], K)), ws.Mc[lv - 1])
        lref = ws.L if slot == 0 else ws.S[lv]
        assert np.array_equal(unpack_digits(w.Lcat[slot]), lref)
        off = sum(gproto.padded_k(c) for c in w.slot_ranks[:slot])
        assert np.array_equal(unpack_digits(Digits(w.Bx.buf[:K], ri, off)), ws.Nc[lv - 1])
        assert np.array_equal(unpack_digits(Digits(w.Bx.buf[K:], ri, off)), ws.J[lv - 1])

    # Init X
    assert np.array_equal(unpack_digits(buf.rho[0]), cs.R.T)
    for slot, lv in enumerate(w.slot_levels[1:], start=1):
        assert np.array_equal(unpack_digits(buf.rho[slot]), cs.T[lv].T)
    UK = to_np_u32(buf.UK)
    assert np.array_equal(UK[:, :K], ring_sub(cs.U_x, cs.E_x).T)
    assert np.array_equal(UK[:, K:], cs.K.T)

    # mask, server, unmask
    assert np.array_equal(unpack_digits(buf.A_masked), ref.X_masked.T)
    YQ = to_np_u32(buf.YQ)
    assert np.array_equal(YQ[:, :N], ref.Y_masked.T)
    for slot, lv in enumerate(w.slot_levels):
        c0 = w.q_cols[slot]
        assert np.array_equal(YQ[:, c0:c0 + params.ranks[lv - 1]], ref.Q[lv - 1].T)
    Y = buf.Y.cpu().numpy()
    assert np.array_equal(Y, lift(ref.Y).T)

    # the exact identity: Y = (A + E_a)(W + E_w)^T over the ring
    ident = ring_matmul(ring_add(to_ring(A), cs.E_x.T), ring_add(to_ring(W), ws.E_w).T)
    assert np.array_equal(Y.view(np.uint32), ident)
    if params.noise.kind == "zero":
        assert np.array_equal(Y.astype(np.int64), A.astype(np.int64) @ W.astype(np.int64).T)
    return Y


@pytest.mark.parametrize("params", [PARAMS_D1_SMALL_R128, PARAMS_D2_SPARSE, PARAMS_D3_SPARSE_SMALL],
                         ids=["d1-small", "d2-sparse", "d3-sparse-small"])
def test_single_masked_matmul_workload(params):
    A, W = int8_operands(SMALL_CASE["M"], SMALL_CASE["K"], SMALL_CASE["N"], SMALL_CASE["seed"])
    Y = _check_run(A, W, params, SEED)
    # protocol error is small: |Y - A W^T| of order sigma sqrt(||a||^2 + ||w||^2)
    err = Y.astype(np.int64) - A.astype(np.int64) @ W.astype(np.int64).T
    if params.noise.kind == "zero":
        assert np.all(err == 0)
    else:
        assert np.abs(err).max() < 20 * 0.5 * np.sqrt(2 * 512 * 127 ** 2 / 3)


@pytest.mark.parametrize("M,K,N,ranks", [(37, 200, 150, (96,)), (130, 333, 70, (64, 32)), (1, 64, 64, (64,))])
def test_ragged_shapes(M, K, N, ranks):
    rng = np.random.default_rng(M + K + N)
    A = rng.integers(-127, 128, (M, K), dtype=np.int8)
    W = rng.integers(-127, 128, (N, K), dtype=np.int8)
    p = ProtocolParams(ranks=ranks, noise=NoiseSpec("dgauss", 0.5, 4), sparse_log2_inv_density=3)
    _check_run(A, W, p, SEED + M)


def test_mask_invariance_on_gpu():
    """With E = 0 different seeds unmask to the same plaintext product."""
    A, W = int8_operands(64, 512, 512, 0)
    p = PARAMS_D2_SPARSE
    ref = A.astype(np.int64) @ W.astype(np.int64).T
    for seed in (1, 99, 0xFFFF_FFFF_0000_0001):
        w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), p, seed, 3)
        buf = gproto.run_call(w, torch.from_numpy(A).cuda(), 5)
        torch.cuda.synchronize()
        assert np.array_equal(buf.Y.cpu().numpy().astype(np.int64), ref)


@pytest.mark.parametrize("M,K,N,ranks", [(1, 64, 64, (64,)), (5, 200, 152, (96, 32)), (16, 128, 260, (64,)),
                                         (3, 96, 150, (64,)), (17, 64, 64, (64,))])
def test_unmask_form_by_token_count(monkeypatch, M, K, N, ranks):
    """Up to 16 tokens, with Q's columns of [Y' | Q] 16-byte aligned (N a
    multiple of 4), unmasking reads Q as ring words (mosaic_unmask_words,
    no conversion pass); otherwise Q is converted to digits first. Both
    give the oracle's Y (every intermediate checked by _check_run)."""
    calls = {"words": 0, "digits": 0}
    words, digits = gproto.m.mosaic_unmask_words, gproto.m.mosaic_unmask

    def count_words(*a, **k):
        calls["words"] += 1
        return words(*a, **k)

    def count_digits(*a, **k):
        if a[2] is not None:                    # a product term (not the dequantisation-only form)
            calls["digits"] += 1
        return digits(*a, **k)
    monkeypatch.setattr(gproto.m, "mosaic_unmask_words", count_words)
    monkeypatch.setattr(gproto.m, "mosaic_unmask", count_digits)
    rng = np.random.default_rng(7 * M + N)
    A = rng.integers(-127, 128, (M, K), dtype=np.int8)
    W = rng.integers(-127, 128, (N, K), dtype=np.int8)
    p = ProtocolParams(ranks=ranks, noise=NoiseSpec("dgauss", 0.5, 4), sparse_log2_inv_density=3)
    _check_run(A, W, p, SEED + 3 * M)
    expect_words = M <= 16 and N % 4 == 0
    assert calls == {"words": int(expect_words), "digits": int(not expect_words)}
