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
                              PREFILL_KN, PREFILL_SEED, int8_operands)
from tests.gpu_util import to_np_u32

pytestmark = pytest.mark.gpu

PARAMS = {"d1": PARAMS_D1_SMALL_R128, "d2": PARAMS_D2_SPARSE, "d3": PARAMS_D3_SPARSE_SMALL}


def _add_host(t: torch.Tensor, i: int, j: int, delta: int) -> None:
    """t[i, j] += delta (mod 2^32), done on the host and copied back."""
    v = int(t[i, j].item()) & 0xFFFFFFFF
    t[i, j] = np.uint32((v + delta) % 2 ** 32).view(np.int32).item()


@pytest.mark.parametrize("name", ["d1", "d2", "d3"])
@pytest.mark.parametrize("N", [512, 516, 510], ids=["one-call", "words", "digit-copies"])
def test_check_sides_match_oracle(name, N):
    """Both sides of the check against the oracle, with rhs formed from
    [Y' | Q] as ring words (N a multiple of 4) or through digit copies
    (N = 510); at N = 512 the one-call check (d = lhs - rhs) is also run and
    must return an all-zero d."""
    p = PARAMS[name]
    A, W = int8_operands(64, 512, N, 0)
    seed, t = 4321, 8
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), p, seed, weight_id=2, check_vectors=t)
    buf = gproto.run_call(w, torch.from_numpy(A).cuda(), call_id=9)
    count = gproto.verify(w, 64, buf, sides=True)
    torch.cuda.synchronize()
    assert int(count.item()) == 0
    res = oproto.run(A, W, p, seed, weight_id=2, call_id=9)
    aW, aQ = integ.check_vectors(t, N, list(p.ranks), seed, 2)
    cT = integ.key(aW, aQ, res.ws.W_masked, {i + 1: mc for i, mc in enumerate(res.ws.Mc)})
    lhs, rhs = integ.sides(cT, aW, aQ, res.X_masked.T, res.Y_masked.T.copy(),
                           {i + 1: q.T.copy() for i, q in enumerate(res.Q)})
    assert np.array_equal(to_np_u32(buf.check[0]), lhs)
    assert np.array_equal(to_np_u32(buf.check[1]), rhs)
    assert np.array_equal(lhs, rhs)
    if N % 64 == 0:
        assert int(gproto.verify(w, 64, buf).item()) == 0
        assert not np.any(to_np_u32(buf.check_diff))


def _check_column_vectors(w, aW, aQ, col):
    """The check vectors' column that multiplies column col of [Y' | Q]."""
    if col < w.N:
        return aW[:, col]
    for slot, lv in enumerate(w.slot_levels):
        c0 = w.q_cols[slot]
        if c0 <= col < c0 + aQ[lv].shape[1]:
            return aQ[lv][:, col - c0]
    return np.zeros(aW.shape[0], dtype=np.uint32)           # a padding column of Q


@pytest.mark.parametrize("name", ["d1", "d2", "d3"])
def test_check_difference_matches_oracle(name):
    """The one-call check after several outputs were changed: d equals, for
    every (vector, token), minus the sum over that token's changed columns of
    the vector's entry times the change, computed from the oracle's check
    vectors; count is the number of nonzero entries of d."""
    p = PARAMS[name]
    A, W = int8_operands(64, 512, 512, 1)
    seed, t = 555, 12
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), p, seed, weight_id=3, check_vectors=t)
    buf = gproto.run_call(w, torch.from_numpy(A).cuda(), call_id=4)
    torch.cuda.synchronize()
    aW, aQ = integ.check_vectors(t, 512, list(p.ranks), seed, 3)
    last = w.q_cols[-1]
    changes = [(5, 17, 1), (5, 512 + 3, 0x12345), (40, 511, 1 << 31), (63, last, 7), (63, 0, 2 ** 32 - 7)]
    expect = np.zeros((t, 64), dtype=np.uint64)
    for i, col, delta in changes:
        _add_host(buf.YQ, i, col, delta)
        a = _check_column_vectors(w, aW, aQ, col).astype(np.uint64)
        expect[:, i] = (expect[:, i] + (2 ** 32 - (a * delta) % 2 ** 32)) % 2 ** 32
    got = int(gproto.verify(w, 64, buf).item())
    d = to_np_u32(buf.check_diff)
    assert np.array_equal(d, expect.astype(np.uint32))
    assert got == int(np.count_nonzero(expect)) > 0


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


@pytest.mark.parametrize("shape_id", range(len(PREFILL_KN)), ids=[f"{k}x{n}" for k, n in PREFILL_KN])
def test_full_size_prefill_check(shape_id):
    """M = 2048 at the three prefill shapes, rank 1536, 32 check vectors:
    honest outputs pass; an odd error in one Y' entry, then in one Q entry,
    is caught by every vector."""
    K, N = PREFILL_KN[shape_id]
    M, t = 2048, 32
    A, W = int8_operands(M, K, N, PREFILL_SEED)
    seed = 0x6D6F736169630000 | PREFILL_SEED
    print(f"integrity check at 2048 x {K} x {N}", flush=True)
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), PARAMS_PAPER_D1, seed, weight_id=shape_id, check_vectors=t)
    buf = gproto.run_call(w, torch.from_numpy(A).cuda(), call_id=1)
    assert int(gproto.verify(w, M, buf).item()) == 0
    aW, aQ = integ.check_vectors(t, N, [1536], seed, shape_id)
    _add_host(buf.YQ, 1000, N - 7, 3)
    got = int(gproto.verify(w, M, buf).item())
    assert got == sum(1 for j in range(t) if (int(aW[j, N - 7]) * 3) % 2 ** 32 != 0) == t
    _add_host(buf.YQ, 1000, N - 7, 2 ** 32 - 3)                     # undo
    assert int(gproto.verify(w, M, buf).item()) == 0
    _add_host(buf.YQ, 2047, w.q_cols[0] + 1535, 5)
    got = int(gproto.verify(w, M, buf).item())
    assert got == sum(1 for j in range(t) if (int(aQ[1][j, 1535]) * 5) % 2 ** 32 != 0) == t


def test_check_graph_replay():
    """The check captured in a HIP graph and replayed with the server's
    outputs changed on the host between replays: each replay's count equals
    the eager check's on the same outputs."""
    p = PARAMS_D1_SMALL_R128
    A, W = int8_operands(64, 512, 512, 5)
    t = 16
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), p, 99, weight_id=4, check_vectors=t)
    buf = gproto.run_call(w, torch.from_numpy(A).cuda(), call_id=2)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        count = gproto.verify(w, 64, buf)
    for rep, (i, j, delta) in enumerate([(0, 0, 0), (7, 300, 1), (7, 300, 2 ** 32 - 1), (63, 512 + 9, 1 << 31)]):
        if delta:
            _add_host(buf.YQ, i, j, delta)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = int(count.item())
        eager = int(gproto.verify(w, 64, buf).item())
        assert got == eager, rep
    assert got > 0


@pytest.mark.parametrize("rows,cols,ld", [(1, 1, 1), (3, 5, 8), (32, 2048, 2048), (64, 2049, 2051),
                                          (4096, 4100, 4101)])
def test_count_mismatches(rows, cols, ld):
    """Differing entries counted over every element, in one workgroup up to
    grids that stride (4096 x 4100: more 4-column groups than 1024
    workgroups of 256 threads cover at once); entries past cols differ in
    every row and must not be counted. The count starts non-zero."""
    from paper_2607_29221_amd import mosaic as m
    rng = np.random.default_rng(rows * 31 + cols)
    a = rng.integers(0, 2 ** 32, (rows, ld), dtype=np.uint64).astype(np.uint32)
    b = a.copy()
    b[:, cols:] ^= 1
    flip = rng.random((rows, cols)) < 0.01
    flip[rows - 1, cols - 1] = True
    b[:, :cols][flip] += np.uint32(1 << 31)
    da = torch.from_numpy(a.view(np.int32)).cuda()[:, :cols]
    db = torch.from_numpy(b.view(np.int32)).cuda()[:, :cols]
    count = torch.full((1,), 12345, dtype=torch.int64, device="cuda")
    m.mosaic_count_mismatches(da, db, count)
    torch.cuda.synchronize()
    assert int(count.item()) == int(flip.sum())


@pytest.mark.parametrize("M,K,N,t", [(16, 33000, 512, 1), (5, 64, 32768, 64), (1, 4096, 4096, 32)],
                         ids=["key-chunks-t1", "check-chunks-t64", "one-token"])
def test_check_chunks_and_vector_counts(M, K, N, t):
    """The one-call check where an inner dimension exceeds one launch's range
    (K = 33000: the key product in two chunks; N + R = 32896: the check
    product in two chunks), with 1 and 64 check vectors and for one token:
    honest outputs give an all-zero d; one changed output is caught by the
    vectors whose entry times the change is non-zero, and d holds exactly
    that column's entries."""
    p = PARAMS_D1_SMALL_R128
    A, W = int8_operands(M, K, N, 9)
    seed = 31337
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), p, seed, weight_id=5, check_vectors=t)
    buf = gproto.run_call(w, torch.from_numpy(A).cuda(), call_id=3)
    assert int(gproto.verify(w, M, buf).item()) == 0
    assert not np.any(to_np_u32(buf.check_diff))
    aW, _ = integ.check_vectors(t, N, list(p.ranks), seed, 5)
    col, delta = N - 1, 0x01000001
    _add_host(buf.YQ, M - 1, col, delta)
    got = int(gproto.verify(w, M, buf).item())
    expect = np.zeros((t, M), dtype=np.uint64)
    expect[:, M - 1] = (2 ** 32 - (aW[:, col].astype(np.uint64) * delta) % 2 ** 32) % 2 ** 32
    assert np.array_equal(to_np_u32(buf.check_diff), expect.astype(np.uint32))
    assert got == int(np.count_nonzero(expect[:, M - 1]))
