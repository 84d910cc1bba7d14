"""Integrity check of the server's outputs (Freivalds' test) through the
C ABI: both sides of the check equal the oracle's bit for bit, honest calls
are accepted, and an output corrupted on the host side is caught exactly as
often as the check vectors predict."""
import numpy as np
import pytest
import torch

from oracle import integrity as integ
from oracle import protocol as oproto
from paper_2607_29221_amd import protocol as gproto
from synthetic_inputs import (PARAMS_D1_SMALL_R128, PARAMS_D2_SPARSE, PARAMS_D3_SPARSE_SMALL, PARAMS_PAPER_D1,
                              PREFILL_SEED, int8_operands)
from tests.gpu_util import to_np_u32

pytestmark = pytest.mark.gpu

PARAMS = {"d1": PARAMS_D1_SMALL_R128, "d2": PARAMS_D2_SPARSE, "d3": PARAMS_D3_SPARSE_SMALL}


def _add_host(t: torch.Tensor, i: int, j: int, delta: int) -> None:
    """t[i, j] += delta (mod 2^32), done on the host and copied back."""
    v = int(t[i, j].item()) & 0xFFFFFFFF
    t[i, j] = np.uint32((v + delta) % 2 ** 32).view(np.int32).item()


@pytest.mark.parametrize("name", ["d1", "d2", "d3"])
def test_check_sides_match_oracle(name):
    p = PARAMS[name]
    A, W = int8_operands(64, 512, 512, 0)
    seed, t = 4321, 8
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), p, seed, weight_id=2, check_vectors=t)
    buf = gproto.run_call(w, torch.from_numpy(A).cuda(), call_id=9)
    count = gproto.verify(w, 64, buf)
    torch.cuda.synchronize()
    assert int(count.item()) == 0
    res = oproto.run(A, W, p, seed, weight_id=2, call_id=9)
    aW, aQ = integ.check_vectors(t, 512, list(p.ranks), seed, 2)
    cT = integ.key(aW, aQ, res.ws.W_masked, {i + 1: mc for i, mc in enumerate(res.ws.Mc)})
    lhs, rhs = integ.sides(cT, aW, aQ, res.X_masked.T, res.Y_masked.T.copy(),
                           {i + 1: q.T.copy() for i, q in enumerate(res.Q)})
    assert np.array_equal(to_np_u32(buf.check[0]), lhs)
    assert np.array_equal(to_np_u32(buf.check[1]), rhs)
    assert np.array_equal(lhs, rhs)


@pytest.mark.parametrize("delta", [1, 0x10000, 1 << 31])
def test_corrupted_outputs_detected(delta):
    """One entry of Y' and then one entry of Q_d is changed by delta after
    the server product; the mismatch count equals the number of check
    vectors j with a[j, col] * delta != 0 (mod 2^32)."""
    p = PARAMS_D3_SPARSE_SMALL
    A, W = int8_operands(64, 512, 512, 0)
    seed, t = 77, 16
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), p, seed, weight_id=1, check_vectors=t)
    Ad = torch.from_numpy(A).cuda()
    aW, aQ = integ.check_vectors(t, 512, list(p.ranks), seed, 1)

    buf = gproto.alloc_call(w, 64)
    gproto.init_x(w, 64, 3, buf)
    gproto.mask(w, Ad, 3, buf)
    gproto.server(w, 64, buf)
    torch.cuda.synchronize()
    _add_host(buf.YQ, 10, 100, delta)
    got = int(gproto.verify(w, 64, buf).item())
    expect = sum(1 for j in range(t) if (int(aW[j, 100]) * delta) % 2 ** 32 != 0)
    assert got == expect and (delta != 1 or got == t)

    gproto.server(w, 64, buf)                       # fresh honest outputs
    torch.cuda.synchronize()
    assert int(gproto.verify(w, 64, buf).item()) == 0
    lv = w.slot_levels[0]                           # level d, first Q slot
    _add_host(buf.YQ, 63, w.q_cols[0] + 5, delta)
    got = int(gproto.verify(w, 64, buf).item())
    expect = sum(1 for j in range(t) if (int(aQ[lv][j, 5]) * delta) % 2 ** 32 != 0)
    assert got == expect


def test_full_size_prefill_check():
    """M = 2048, K = N = 8192, rank 1536, 32 check vectors: honest outputs
    pass, an odd error in one Y' entry is caught by every vector."""
    K, N, M, t = 8192, 8192, 2048, 32
    A, W = int8_operands(M, K, N, PREFILL_SEED)
    seed = 0x6D6F736169630000 | PREFILL_SEED
    print("integrity check at 2048 x 8192 x 8192", flush=True)
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), PARAMS_PAPER_D1, seed, weight_id=0, check_vectors=t)
    buf = gproto.run_call(w, torch.from_numpy(A).cuda(), call_id=1)
    assert int(gproto.verify(w, M, buf).item()) == 0
    aW, _ = integ.check_vectors(t, N, [1536], seed, 0)
    _add_host(buf.YQ, 1000, 4321, 3)
    got = int(gproto.verify(w, M, buf).item())
    assert got == sum(1 for j in range(t) if (int(aW[j, 4321]) * 3) % 2 ** 32 != 0) == t
