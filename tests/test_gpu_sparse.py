"""Sparse LPN matrices in compressed rows, through the C ABI: the compressed
form equals the oracle's SPARSE stream matrix exactly, the two gather
products equal ring products with that matrix, and the protocol in sparse
mode gives every output of the oracle (and of the dense mode) bit for bit."""
import numpy as np
import pytest
import torch

from oracle import protocol as oproto
from oracle import sampling as smp
from oracle.ring import lift, ring_add, ring_matmul, ring_sub
from paper_2607_29221_amd import mosaic as m
from paper_2607_29221_amd import protocol as gproto
from synthetic_inputs import (PARAMS_D2_SPARSE, PARAMS_D3_SPARSE_SMALL, PARAMS_PAPER_D2_SPARSE,
                              PARAMS_PAPER_D3_SPARSE, DECODE_KN, DECODE_M, DECODE_SEED, NoiseSpec, ProtocolParams,
                              int8_operands)
from tests.gpu_util import noisy_identity, to_dev_ring, to_np_u32

pytestmark = pytest.mark.gpu


def _dense_from_csr(p: m.SparseRows) -> np.ndarray:
    rp = p.row_ptr.cpu().numpy()
    nnz = int(rp[-1])
    ci = p.col_idx.cpu().numpy()[:nnz]
    va = p.values.cpu().numpy().view(np.uint32)[:nnz]
    out = np.zeros((p.rows, p.cols), dtype=np.uint32)
    for i in range(p.rows):
        cols = ci[rp[i]:rp[i + 1]]
        assert np.all(np.diff(cols) > 0)                  # increasing within a row
        out[i, cols] = va[rp[i]:rp[i + 1]]
    return out


@pytest.mark.parametrize("rows,cols,s", [(5, 1536, 6), (300, 70, 2), (5000, 8, 4), (3, 33, 0), (40, 100, 31),
                                         (0, 10, 6), (7, 0, 6), (1, 1, 0)])
@pytest.mark.parametrize("exact", [True, False])
def test_csr_matches_oracle(rows, cols, s, exact):
    seed, stream, inst = 99, 0x41, 3
    p = m.mosaic_sparse_csr(m.rng(seed, stream, inst, m.DIST_SPARSE, log2_inv_density=s), rows, cols, exact=exact)
    ref = smp.sample_matrix("sparse", rows, cols, seed, stream, inst, log2_inv_density=s)
    if rows and cols:
        assert np.array_equal(_dense_from_csr(p), ref)
    rp = p.row_ptr.cpu().numpy()
    assert rp[0] == 0 and rp[-1] == np.count_nonzero(ref) if rows else rp[-1] == 0
    assert np.array_equal(np.diff(rp), np.count_nonzero(ref, axis=1)) if rows else True


@pytest.mark.parametrize("subtract", [False, True])
def test_gather_rows_and_cols(subtract):
    rng = np.random.default_rng(7)
    rows, r, ncols, M = 37, 300, 517, 19
    p = m.mosaic_sparse_csr(m.rng(5, 0x42, 0, m.DIST_SPARSE, log2_inv_density=3), rows, r)
    P = smp.sample_matrix("sparse", rows, r, 5, 0x42, 0, log2_inv_density=3)
    D = rng.integers(0, 2 ** 32, (r, ncols), dtype=np.uint32)
    C0 = rng.integers(0, 2 ** 32, (rows, ncols + 3), dtype=np.uint32)
    c = to_dev_ring(C0)
    m.mosaic_sparse_gather_rows(p, to_dev_ring(D), ncols, c, subtract=subtract)
    prod = ring_matmul(P, D)
    want = C0.copy()
    want[:, :ncols] = ring_sub(C0[:, :ncols], prod) if subtract else ring_add(C0[:, :ncols], prod)
    torch.cuda.synchronize()
    assert np.array_equal(to_np_u32(c), want)

    Dm = rng.integers(0, 2 ** 32, (M, r + 5), dtype=np.uint32)       # M x r with ld > r
    C1 = rng.integers(0, 2 ** 32, (M, rows), dtype=np.uint32)
    c1 = to_dev_ring(C1)
    dm = to_dev_ring(Dm)
    m.mosaic_sparse_gather_cols(p, dm[:, :r], M, c1, subtract=subtract)
    prod = ring_matmul(Dm[:, :r], P.T)
    want = ring_sub(C1, prod) if subtract else ring_add(C1, prod)
    torch.cuda.synchronize()
    assert np.array_equal(to_np_u32(c1), want)

    # the same gather writing the dequantised result too (with and without a
    # bias): y = (c s_rows) s_cols (+ bias), each step rounded to fp32
    for with_bias in (False, True):
        c2 = to_dev_ring(C1)
        sr = torch.rand(M, device="cuda") * 1e-3
        sc = torch.rand(rows, device="cuda") * 1e-3
        bias = torch.randn(rows, device="cuda") if with_bias else None
        yf = torch.full((M, rows + 2), 7.0, device="cuda")
        m.mosaic_sparse_gather_cols(p, dm[:, :r], M, c2, subtract=subtract, y_f32=yf[:, :rows], s_rows=sr,
                                    s_cols=sc, bias=bias)
        torch.cuda.synchronize()
        assert np.array_equal(to_np_u32(c2), want)
        ref = (want.view(np.int32).astype(np.float32) * sr.cpu().numpy()[:, None]) * sc.cpu().numpy()[None, :]
        if with_bias:
            ref = (ref + bias.cpu().numpy()[None, :]).astype(np.float32)
        got = yf.cpu().numpy()
        assert np.array_equal(got[:, :rows], ref)
        assert np.all(got[:, rows:] == 7.0)


@pytest.mark.parametrize("rows,r,ncols,s", [(9, 300, 517, 3), (3, 5000, 70, 0), (4, 5000, 300, 6), (1, 1, 1, 0),
                                            (2, 64, 4096, 31), (40, 700, 2000, 2), (6, 2100, 13000, 0)])
@pytest.mark.parametrize("subtract", [False, True])
def test_stream_gather_rows_and_long_rows(rows, r, ncols, s, subtract):
    """Rows drawn inside the gather, and compressed rows longer than one LDS
    staging chunk (density 1 over 5000 columns); few rows split their entries
    between four waves per 64 columns, 40 x 2000 and 6 x 13000 (more than
    four workgroups per compute unit) take one wave per 64 columns."""
    rng = np.random.default_rng(rows * r + ncols)
    seed, stream, inst = 12, 0x43, 5
    P = smp.sample_matrix("sparse", rows, r, seed, stream, inst, log2_inv_density=s)
    D = rng.integers(0, 2 ** 32, (r, ncols), dtype=np.uint32)
    C0 = rng.integers(0, 2 ** 32, (rows, ncols), dtype=np.uint32)
    prod = ring_matmul(P, D)
    want = ring_sub(C0, prod) if subtract else ring_add(C0, prod)
    rr = m.rng(seed, stream, inst, m.DIST_SPARSE, log2_inv_density=s)
    c = to_dev_ring(C0)
    m.mosaic_sparse_stream_gather_rows(rr, rows, r, to_dev_ring(D), ncols, c, subtract=subtract)
    c2 = to_dev_ring(C0)
    m.mosaic_sparse_gather_rows(m.mosaic_sparse_csr(rr, rows, r), to_dev_ring(D), ncols, c2, subtract=subtract)
    torch.cuda.synchronize()
    assert np.array_equal(to_np_u32(c), want)
    assert np.array_equal(to_np_u32(c2), want)


@pytest.mark.parametrize("M", [1, 3, 4, 5, 16, 17])
@pytest.mark.parametrize("kind", ["sparse", "weight"])
def test_gather_cols_token_blocks(M, kind):
    """The column gather for 1 to 17 rows of d (one workgroup covers all rows
    up to 16), against the oracle's product, with a WEIGHT matrix of 80
    entries per row and a Bernoulli one."""
    rows, r = 1000, 1024
    rng = np.random.default_rng(M * 7 + len(kind))
    if kind == "weight":
        rr = m.rng(44, 0x45, 2, m.DIST_WEIGHT, row_weight=80)
        P = smp.sample_matrix("weight", rows, r, 44, 0x45, 2, row_weight=80)
    else:
        rr = m.rng(44, 0x45, 2, m.DIST_SPARSE, log2_inv_density=4)
        P = smp.sample_matrix("sparse", rows, r, 44, 0x45, 2, log2_inv_density=4)
    p = m.mosaic_sparse_csr(rr, rows, r)
    D = rng.integers(0, 2 ** 32, (M, r + 3), dtype=np.uint32)
    C0 = rng.integers(0, 2 ** 32, (M, rows), dtype=np.uint32)
    c = to_dev_ring(C0)
    m.mosaic_sparse_gather_cols(p, to_dev_ring(D)[:, :r], M, c, subtract=True)
    torch.cuda.synchronize()
    assert np.array_equal(to_np_u32(c), ring_sub(C0, ring_matmul(D[:, :r], P.T)))


@pytest.mark.parametrize("params", [PARAMS_D2_SPARSE, PARAMS_D3_SPARSE_SMALL,
                                    ProtocolParams(ranks=(128, 64), noise=NoiseSpec("dgauss", 0.5, 4),
                                                   sparse_log2_inv_density=2)],
                         ids=["d2", "d3", "d2-dense-lpn-noise"])
@pytest.mark.parametrize("shape", [(64, 512, 512), (70, 130, 200)], ids=["small", "ragged"])
def test_sparse_mode_protocol(params, shape):
    M, K, N = shape
    A, W = int8_operands(M, K, N, 0)
    seed = 31337
    ref = oproto.run(A, W, params, seed, weight_id=1, call_id=2)
    outs = {}
    for sparse in (False, True):
        w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), params, seed, 1, sparse_lpn=sparse)
        buf = gproto.run_call(w, torch.from_numpy(A).cuda(), 2)
        torch.cuda.synchronize()
        outs[sparse] = (to_np_u32(buf.UK), to_np_u32(buf.YQ), buf.Y.cpu().numpy())
    UK, YQ, Y = outs[True]
    cs = ref.cs
    assert np.array_equal(UK[:, :K], ring_sub(cs.U_x, cs.E_x).T)
    assert np.array_equal(UK[:, K:], cs.K.T)
    assert np.array_equal(YQ[:, :N], ref.Y_masked.T)
    assert np.array_equal(Y, lift(ref.Y).T)
    for a, b in zip(outs[False], outs[True]):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("shape_id", range(len(DECODE_KN)), ids=[f"{k}x{n}" for k, n in DECODE_KN])
def test_sparse_mode_decode_exact(shape_id):
    """Decode shapes, depth 2 with ranks (1536, 1024), E = 0, sparse mode:
    Y equals A W^T exactly for every token count."""
    K, N = DECODE_KN[shape_id]
    A, W = int8_operands(max(DECODE_M), K, N, DECODE_SEED)
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), PARAMS_PAPER_D2_SPARSE, 0xDEC0DE00 + shape_id, shape_id,
                            sparse_lpn=True)
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    for Mi in DECODE_M:
        buf = gproto.run_call(w, torch.from_numpy(np.ascontiguousarray(A[:Mi])).cuda(), call_id=Mi)
        torch.cuda.synchronize()
        assert np.array_equal(buf.Y.cpu().numpy().astype(np.float64), ref[:Mi])


@pytest.mark.parametrize("sparse", [True, False])
def test_paper_depth3_decode_exact(sparse):
    """The paper's depth-3 ranks (1536, 1024, 652; the last padded to 704
    digit columns) at the 4096 x 4096 decode shape, E = 0: Y equals A W^T
    exactly for every token count, in sparse and dense mode."""
    K, N = DECODE_KN[0]
    A, W = int8_operands(max(DECODE_M), K, N, DECODE_SEED)
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), PARAMS_PAPER_D3_SPARSE, 0xDEC0DE30, 3, sparse_lpn=sparse)
    ref = A.astype(np.float64) @ W.astype(np.float64).T
    for Mi in DECODE_M:
        buf = gproto.run_call(w, torch.from_numpy(np.ascontiguousarray(A[:Mi])).cuda(), call_id=Mi)
        torch.cuda.synchronize()
        assert np.array_equal(buf.Y.cpu().numpy().astype(np.float64), ref[:Mi])


def test_sparse_mode_dequantised_output():
    """Unmasking with dequantisation in sparse mode (gathers, then an
    elementwise dequantisation) equals the dense mode's fused epilogue."""
    M, K, N = 40, 256, 200
    A, W = int8_operands(M, K, N, 3)
    p = PARAMS_D3_SPARSE_SMALL
    sr = torch.rand(M, device="cuda") * 1e-3
    sc = torch.rand(N, device="cuda") * 1e-3
    outs = []
    for sparse in (False, True):
        w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), p, 5, 1, sparse_lpn=sparse)
        buf = gproto.alloc_call(w, M)
        gproto.init_x(w, M, 4, buf)
        gproto.mask(w, torch.from_numpy(A).cuda(), 4, buf)
        gproto.server(w, M, buf)
        yf = torch.empty((M, N), dtype=torch.float32, device="cuda")
        gproto.unmask(w, M, buf, y_f32=yf, s_rows=sr, s_cols=sc)
        torch.cuda.synchronize()
        outs.append((buf.Y.cpu().numpy(), yf.cpu().numpy()))
    assert np.array_equal(outs[0][0], outs[1][0])
    assert np.array_equal(outs[0][1], outs[1][1])


# --- fixed row weight (Example 4.1: t nonzeros per row) ---

@pytest.mark.parametrize("rows,cols,t", [(5, 1536, 80), (64, 1024, 80), (33, 70, 70), (4, 8192, 2048),
                                         (3, 5, 0), (1, 1, 1), (130, 652, 80),
                                         # rows of up to 256 entries are resolved in parallel: full
                                         # permutations and dense rows (many repeated positions)
                                         (5, 256, 256), (4, 300, 256), (6, 64, 64), (6, 65, 65),
                                         (3, 300, 257)])
def test_weighted_sample_matches_oracle(rows, cols, t):
    """mosaic_sample with a WEIGHT stream: ring words and digits equal the
    oracle's partial-shuffle matrix (zeros elsewhere, padding digits zero)."""
    seed, stream, inst = 77, 0x44, 5
    r = m.rng(seed, stream, inst, m.DIST_WEIGHT, row_weight=t)
    out = torch.full((rows, cols + 3), -1, dtype=torch.int32, device="cuda")
    dig = m.Digits(torch.full((rows, 4 * m.padded_k(cols)), 7, dtype=torch.int8, device="cuda"), cols)
    m.mosaic_sample(r, rows, cols, out=out[:, :cols], out_dig=dig)
    torch.cuda.synchronize()
    ref = smp.sample_matrix("weight", rows, cols, seed, stream, inst, row_weight=t)
    got = to_np_u32(out)
    assert np.array_equal(got[:, :cols], ref)
    assert np.all(got[:, cols:] == 0xFFFFFFFF)
    from tests.gpu_util import pad_is_zero, unpack_digits
    assert np.array_equal(unpack_digits(dig), ref)
    assert pad_is_zero(dig)


@pytest.mark.parametrize("rows,cols,t", [(300, 1536, 80), (17, 1024, 80), (9, 40, 40), (2, 8192, 2048),
                                         (7, 256, 256), (5, 8192, 256)])
def test_weighted_csr_matches_oracle(rows, cols, t):
    """Compressed rows of a WEIGHT stream: row_ptr = i t, and each row lists
    the oracle's columns and values in the order of the shuffle's steps."""
    seed, stream, inst = 8, 0x45, 1
    p = m.mosaic_sparse_csr(m.rng(seed, stream, inst, m.DIST_WEIGHT, row_weight=t), rows, cols)
    torch.cuda.synchronize()
    pos, val = smp.weighted_rows(range(rows), cols, t, seed, stream, inst)
    assert np.array_equal(p.row_ptr.cpu().numpy(), np.arange(rows + 1) * t)
    assert np.array_equal(p.col_idx.cpu().numpy()[: rows * t].reshape(rows, t), pos)
    assert np.array_equal(p.values.cpu().numpy().view(np.uint32)[: rows * t].reshape(rows, t), val)


@pytest.mark.parametrize("rows,r,ncols,t", [(9, 1536, 517, 80), (64, 1024, 8192, 80), (3, 300, 70, 300),
                                            (1, 1, 1, 1), (5, 2048, 300, 2048), (4, 256, 300, 256),
                                            (1, 652, 18432, 80)])
@pytest.mark.parametrize("subtract", [False, True])
def test_weighted_stream_gather(rows, r, ncols, t, subtract):
    """T_{i+1} terms with WEIGHT rows drawn inside the gather, and the same
    through compressed rows, equal ring products with the oracle's matrix."""
    rng = np.random.default_rng(rows + r + t)
    seed, stream, inst = 13, 0x63, 9
    P = smp.sample_matrix("weight", rows, r, seed, stream, inst, row_weight=t)
    D = rng.integers(0, 2 ** 32, (r, ncols), dtype=np.uint32)
    C0 = rng.integers(0, 2 ** 32, (rows, ncols), dtype=np.uint32)
    prod = ring_matmul(P, D)
    want = ring_sub(C0, prod) if subtract else ring_add(C0, prod)
    rr = m.rng(seed, stream, inst, m.DIST_WEIGHT, row_weight=t)
    c = to_dev_ring(C0)
    m.mosaic_sparse_stream_gather_rows(rr, rows, r, to_dev_ring(D), ncols, c, subtract=subtract)
    c2 = to_dev_ring(C0)
    m.mosaic_sparse_gather_rows(m.mosaic_sparse_csr(rr, rows, r), to_dev_ring(D), ncols, c2, subtract=subtract)
    torch.cuda.synchronize()
    assert np.array_equal(to_np_u32(c), want)
    assert np.array_equal(to_np_u32(c2), want)


def test_weighted_rejected_where_unsupported():
    r = m.rng(1, 2, 3, m.DIST_WEIGHT, row_weight=5)
    out = torch.empty((4, 4), dtype=torch.int32, device="cuda")
    with pytest.raises(m.MosaicError):                           # t > cols
        m.mosaic_sample(r, 4, 4, out=out)
    with pytest.raises(m.MosaicError):                           # not drawn inside the mask pass
        m.mosaic_mask(None, out, r, 4, 4, out=out)
    rt = m.rng(1, 2, 3, m.DIST_WEIGHT, row_weight=1, transposed=True)
    with pytest.raises(m.MosaicError):
        m.mosaic_sample(rt, 4, 4, out=out)


@pytest.mark.parametrize("mode", [False, True, None], ids=["dense", "sparse", "auto"])
@pytest.mark.parametrize("shape", [(64, 512, 512), (70, 130, 200), (5, 256, 96)], ids=["small", "ragged", "few"])
def test_weighted_protocol_modes(mode, shape):
    """Depth 3 with fixed row weights, every LPN form: U_a, K_c, Y', Y equal
    the oracle bit for bit."""
    from synthetic_inputs import PARAMS_D3_WEIGHT_SMALL
    M, K, N = shape
    A, W = int8_operands(M, K, N, 4)
    seed = 4242
    ref = oproto.run(A, W, PARAMS_D3_WEIGHT_SMALL, seed, weight_id=2, call_id=3)
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), PARAMS_D3_WEIGHT_SMALL, seed, 2, sparse_lpn=mode)
    buf = gproto.run_call(w, torch.from_numpy(A).cuda(), 3)
    torch.cuda.synchronize()
    UK, YQ = to_np_u32(buf.UK), to_np_u32(buf.YQ)
    cs = ref.cs
    assert np.array_equal(UK[:, :K], ring_sub(cs.U_x, cs.E_x).T)
    assert np.array_equal(UK[:, K:], cs.K.T)
    assert np.array_equal(YQ[:, :N], ref.Y_masked.T)
    assert np.array_equal(buf.Y.cpu().numpy(), lift(ref.Y).T)


@pytest.mark.parametrize("shape_id", range(len(DECODE_KN)), ids=[f"{k}x{n}" for k, n in DECODE_KN])
@pytest.mark.parametrize("which", ["d2-noisy", "paper-d3-t80"])
def test_decode_noisy_exact(shape_id, which):
    """Decode shapes with the paper's LWE error sigma = 0.5: depth 2 (1536,
    1024) at density 2^-6, and Example 4.1 in full (1536, 1024, 652 with
    t = 80). Every output of Y equals (A + E_a)(W + E_w)^T mod 2^32 for
    1, 8 and 64 tokens (sparse calls below 17 tokens, dense above)."""
    from synthetic_inputs import PARAMS_DECODE_D2_NOISY, PARAMS_PAPER_D3_T80
    params = PARAMS_DECODE_D2_NOISY if which == "d2-noisy" else PARAMS_PAPER_D3_T80
    K, N = DECODE_KN[shape_id]
    A, W = int8_operands(max(DECODE_M), K, N, DECODE_SEED)
    seed = 0xDEC0DE50 + shape_id
    w = gproto.MaskedWeight(torch.from_numpy(W).cuda(), params, seed, shape_id)
    for Mi in DECODE_M:
        Ai = np.ascontiguousarray(A[:Mi])
        buf = gproto.run_call(w, torch.from_numpy(Ai).cuda(), call_id=100 + Mi)
        torch.cuda.synchronize()
        want = noisy_identity(Ai, W, params, seed, shape_id, 100 + Mi)
        assert np.array_equal(to_np_u32(buf.Y), want), (which, K, N, Mi)
