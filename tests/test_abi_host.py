"""Host-side checks of the C ABI (no GPU needed): the built library loads,
exports every function the headers under include/ declare, rejects invalid
arguments before launching anything (these run only where no GPU is
present), and computes the same sampler thresholds as the oracle."""
import ctypes
import os
import re

import pytest

from oracle.sampling import dgauss_thresholds
from paper_2607_29221_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mosaic.h")
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]

INVALID, UNSUPPORTED = -1, -2

FAKE = 1 << 20      # an aligned non-null address; never dereferenced on these paths

# The validation tests below hand the entry points a fake device address and
# expect a rejection before any launch. They belong to the CPU build: where a
# GPU is present, a regression in the validation would launch a kernel on
# that address, so they do not run there.
cpu_only = pytest.mark.skipif(os.path.exists("/dev/kfd"),
                              reason="fake-pointer validation tests run only where no GPU is present")


def _declared():
    text = "\n".join(open(h).read() for h in HEADERS)
    return sorted(set(re.findall(r"^\s*(?:mosaic_status|int32_t|const char\*)\s+(mosaic_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(_lib.EXPORTED)


def test_library_matches_sources():
    """The in-tree library was built from the sources in the tree."""
    assert _lib.stale_reason() is None


def test_stale_library_is_refused(monkeypatch):
    """A library whose recorded source digest differs from the sources is
    not loaded (it would run other kernels than the tree holds)."""
    from paper_2607_29221_amd import build
    monkeypatch.setattr(build, "source_digest", lambda: "0" * 64)
    monkeypatch.setattr(_lib, "_lib", None)
    assert "changed after the last build" in _lib.stale_reason()
    with pytest.raises(RuntimeError, match="stale"):
        _lib.load()


def test_abi_version(lib):
    m = re.search(r"#define MOSAIC_ABI_VERSION (\d+)", open(HEADER).read())
    assert lib.mosaic_abi_version() == int(m.group(1))


@pytest.mark.parametrize("sigma,bound", [(0.5, 4), (1.0, 8), (0.0, 4), (3.2, 15), (0.25, 2), (2.0, 1)])
def test_dgauss_thresholds_match_oracle(lib, sigma, bound):
    arr = (ctypes.c_uint64 * (2 * bound))()
    assert lib.mosaic_dgauss_thresholds(sigma, bound, arr) == 0
    assert [int(v) for v in arr] == dgauss_thresholds(sigma, bound)


def test_dgauss_thresholds_rejects(lib):
    arr = (ctypes.c_uint64 * 40)()
    assert lib.mosaic_dgauss_thresholds(0.5, 16, arr) == INVALID
    assert lib.mosaic_dgauss_thresholds(-1.0, 4, arr) == INVALID
    assert lib.mosaic_dgauss_thresholds(float("nan"), 4, arr) == INVALID
    assert lib.mosaic_dgauss_thresholds(0.5, 4, None) == INVALID





@cpu_only
def test_mask_validation(lib):
    r = _lib.MosaicRng(seed=1, stream=2, instance=3, dist=1)
    # no output
    assert lib.mosaic_mask(None, 0, 0, 0, None, 0, ctypes.byref(r), 4, 4, None, 0, None, 0, None) == INVALID
    # bad pitch (must be a multiple of 64 and >= 4 * padded K)
    assert lib.mosaic_mask(None, 0, 0, 0, None, 0, ctypes.byref(r), 4, 100, None, 0, FAKE, 256, None) == INVALID
    assert lib.mosaic_mask(None, 0, 0, 0, None, 0, ctypes.byref(r), 4, 100, None, 0, FAKE, 520, None) == INVALID
    # misaligned digits
    assert lib.mosaic_mask(None, 0, 0, 0, None, 0, ctypes.byref(r), 4, 64, None, 0, FAKE + 8, 256, None) == INVALID
    # ldu / ldo too small, bad dtype, negative size
    assert lib.mosaic_mask(None, 0, 0, 0, FAKE, 3, None, 4, 4, FAKE, 4, None, 0, None) == INVALID
    assert lib.mosaic_mask(None, 0, 0, 0, None, 0, None, 4, 4, FAKE, 3, None, 0, None) == INVALID
    assert lib.mosaic_mask(FAKE, 9, 4, 1, None, 0, None, 4, 4, FAKE, 4, None, 0, None) == INVALID
    assert lib.mosaic_mask(None, 0, 0, 0, None, 0, None, -1, 4, FAKE, 4, None, 0, None) == INVALID
    # bad distributions
    for bad in (_lib.MosaicRng(dist=7), _lib.MosaicRng(dist=2, bound=16, sigma=0.5),
                _lib.MosaicRng(dist=2, bound=4, sigma=-1.0), _lib.MosaicRng(dist=3, log2_inv_density=32)):
        assert lib.mosaic_mask(None, 0, 0, 0, None, 0, ctypes.byref(bad), 4, 4, FAKE, 4, None, 0, None) == INVALID
    assert len(lib.mosaic_last_error_message()) > 0


@cpu_only
def test_matmul_validation(lib):
    # a pitch too small for K (long K itself is accepted: it runs in chunks)
    assert lib.mosaic_masked_matmul(FAKE, 4 * 32768 - 64, FAKE, 4 * 32768, 1, 1, 32768, FAKE, 1, None) == INVALID
    assert lib.mosaic_masked_matmul(FAKE, 256, FAKE, 256, 1, 1, 64, None, 1, None) == INVALID
    assert lib.mosaic_masked_matmul(FAKE, 256, FAKE, 256, 1, 2, 64, FAKE, 1, None) == INVALID   # ldc < N
    assert lib.mosaic_masked_matmul(FAKE, 192, FAKE, 256, 1, 1, 64, FAKE, 1, None) == INVALID   # pitch
    assert lib.mosaic_masked_matmul(None, 256, FAKE, 256, 1, 1, 64, FAKE, 1, None) == INVALID
    assert lib.mosaic_masked_matmul(FAKE, 256, FAKE, 256, -1, 1, 64, FAKE, 1, None) == INVALID


@cpu_only
def test_unmask_validation(lib):
    args = dict(ym=FAKE, ldy=8, kc=None, ldk=0, q=FAKE, qp=256, l=FAKE, lp=256, M=2, N=8, R=64,
                y=FAKE, ldo=8, sr=None, sc=None, bias=None, yf=None, ldf=0)

    def call(**kw):
        a = dict(args, **kw)
        return lib.mosaic_unmask(a["ym"], a["ldy"], a["kc"], a["ldk"], a["q"], a["qp"], a["l"], a["lp"], a["M"],
                                 a["N"], a["R"], a["y"], a["ldo"], a["sr"], a["sc"], a["bias"], a["yf"], a["ldf"],
                                 None)
    assert call(ym=None) == INVALID
    assert call(y=None) == INVALID
    assert call(ldy=7) == INVALID
    assert call(kc=FAKE, ldk=4) == INVALID
    assert call(qp=128) == INVALID
    assert call(l=None) == INVALID
    assert call(yf=FAKE, ldf=8) == INVALID          # fp32 output without scales
    assert call(bias=FAKE) == INVALID               # bias without the fp32 output
    assert call(R=40000, qp=4 * 40000 + 64, lp=4 * 40000 + 64) == UNSUPPORTED


@cpu_only
def test_unmask_words_validation(lib):
    """Q as ring words: the mosaic_unmask rules plus at most 16 rows, q
    16-byte aligned with ldq >= R a multiple of 4."""
    args = dict(ym=FAKE, ldy=8, kc=None, ldk=0, q=FAKE, ldq=64, l=FAKE, lp=256, M=2, N=8, R=64,
                y=FAKE, ldo=8, sr=None, sc=None, bias=None, yf=None, ldf=0)

    def call(**kw):
        a = dict(args, **kw)
        return lib.mosaic_unmask_words(a["ym"], a["ldy"], a["kc"], a["ldk"], a["q"], a["ldq"], a["l"], a["lp"],
                                       a["M"], a["N"], a["R"], a["y"], a["ldo"], a["sr"], a["sc"], a["bias"],
                                       a["yf"], a["ldf"], None)
    assert call(M=17) == UNSUPPORTED
    assert call(ym=None) == INVALID
    assert call(y=None) == INVALID
    assert call(ldy=7) == INVALID
    assert call(q=None) == INVALID
    assert call(ldq=60) == INVALID                  # ldq < R
    assert call(q=FAKE + 4) == UNSUPPORTED          # not 16-byte aligned
    assert call(ldq=66) == UNSUPPORTED              # rows not 16-byte aligned
    assert call(lp=128) == INVALID
    assert call(l=None) == INVALID
    assert call(yf=FAKE, ldf=8) == INVALID
    assert call(bias=FAKE) == INVALID
    assert call(R=40000, ldq=40000, lp=4 * 40000 + 64) == UNSUPPORTED


@cpu_only
def test_hadamard28_validation(lib):
    def call(x=FAKE, ldx=28672, y=FAKE + (1 << 24), ldy=28672, rows=2, n=28672, signs=None, inv=0):
        return lib.mosaic_hadamard28_rotate(x, ldx, y, ldy, rows, n, signs, inv, None)
    assert call(n=28 * 100, ldx=2800, ldy=2800) == UNSUPPORTED   # b not a power of two
    assert call(n=28 * 2048, ldx=57344, ldy=57344) == UNSUPPORTED
    assert call(n=28 * 128, ldx=3584, ldy=3584) == UNSUPPORTED
    assert call(n=1000, ldx=1000, ldy=1000) == UNSUPPORTED        # not 28 b
    assert call(ldx=28670) == INVALID
    assert call(x=FAKE + 4) == INVALID                            # misaligned
    assert call(y=FAKE + 64) == INVALID                           # overlapping, not in place
    assert call(y=FAKE, ldy=28676) == INVALID                     # in place with different ld
    assert call(x=None) == INVALID
    assert call(signs=FAKE + 2) == INVALID
    assert call(rows=0) == 0 and call(rows=-1) == INVALID


@cpu_only
def test_count_mismatches_validation(lib):
    assert lib.mosaic_count_mismatches(FAKE, 4, FAKE, 4, 2, 4, None, None) == INVALID      # no count
    assert lib.mosaic_count_mismatches(None, 4, FAKE, 4, 2, 4, FAKE, None) == INVALID
    assert lib.mosaic_count_mismatches(FAKE, 3, FAKE, 4, 2, 4, FAKE, None) == INVALID      # lda < cols
    assert lib.mosaic_count_mismatches(FAKE, 4, FAKE, 3, 2, 4, FAKE, None) == INVALID
    assert lib.mosaic_count_mismatches(FAKE, 4, FAKE, 4, -1, 4, FAKE, None) == INVALID


@cpu_only
def test_integrity_check_validation(lib):
    def call(ct=FAKE, a=FAKE, a_pitch=256, v=FAKE, yq=FAKE, ldyq=64, t=4, M=4, K=64, NR=64, d=FAKE, ldd=4,
             count=FAKE):
        return lib.mosaic_integrity_check(ct, 256, a, a_pitch, v, 256, yq, ldyq, t, M, K, NR, d, ldd, count, None)
    assert call(count=None) == INVALID
    assert call(t=65) == UNSUPPORTED
    assert call(M=-1) == INVALID
    assert call(d=None) == INVALID
    assert call(ldd=3) == INVALID
    assert call(ct=FAKE + 1) == INVALID
    assert call(a_pitch=192) == INVALID
    assert call(yq=None) == INVALID
    assert call(ldyq=60) == INVALID
    assert call(yq=FAKE + 4) == UNSUPPORTED
    assert call(ldyq=66) == UNSUPPORTED
    assert call(a_pitch=1 << 24) == UNSUPPORTED


@cpu_only
def test_hadamard_validation(lib):
    def call(x=FAKE, ldx=64, y=FAKE + (1 << 24), ldy=64, rows=2, n=64, block=64, signs=None, inv=0):
        return lib.mosaic_hadamard_rotate(x, ldx, y, ldy, rows, n, block, signs, inv, None)
    assert call(block=48) == UNSUPPORTED
    assert call(block=8) == UNSUPPORTED
    assert call(block=65536, n=65536, ldx=65536, ldy=65536) == UNSUPPORTED
    assert call(n=96, block=64, ldx=96, ldy=96) == INVALID      # n not a multiple of block
    assert call(ldx=62) == INVALID
    assert call(x=FAKE + 4) == INVALID                           # misaligned
    assert call(y=FAKE + 64) == INVALID                          # overlapping, not in place
    assert call(y=FAKE, ldy=128, ldx=64) == INVALID              # in place with different ld
    assert call(x=None) == INVALID


@cpu_only
def test_quantize_validation(lib):
    assert lib.mosaic_quantize_rows(FAKE, 8, 2, 8, 0, FAKE, 8, None, 0, None, None) == INVALID
    assert lib.mosaic_quantize_rows(FAKE, 8, 2, 8, 127, None, 0, None, 0, None, None) == INVALID
    assert lib.mosaic_quantize_rows(FAKE, 8, 2, 8, 127, FAKE, 4, None, 0, None, None) == INVALID
    assert lib.mosaic_quantize_rows(FAKE, 8, 2, 8, 127, None, 0, FAKE, 64, None, None) == INVALID


@cpu_only
def test_signs_validation(lib):
    r = _lib.MosaicRng(seed=1)
    assert lib.mosaic_sample_signs(ctypes.byref(r), 8, None, None) == INVALID
    assert lib.mosaic_sample_signs(None, 8, FAKE, None) == INVALID
    assert lib.mosaic_sample_signs(ctypes.byref(r), -1, FAKE, None) == INVALID


def test_zero_sized_calls_are_noops(lib):
    r = _lib.MosaicRng(seed=1, dist=1)
    assert lib.mosaic_mask(None, 0, 0, 0, None, 0, ctypes.byref(r), 0, 5, None, 0, None, 0, None) == 0
    assert lib.mosaic_mask(None, 0, 0, 0, None, 0, ctypes.byref(r), 5, 0, None, 0, None, 0, None) == 0
    assert lib.mosaic_sample(ctypes.byref(r), 0, 0, None, 0, None, 0, None) == 0
    assert lib.mosaic_masked_matmul(None, 0, None, 0, 0, 7, 64, None, 7, None) == 0
    assert lib.mosaic_masked_matmul(None, 0, None, 0, 7, 0, 64, None, 0, None) == 0
    assert lib.mosaic_unmask(None, 0, None, 0, None, 0, None, 0, 0, 4, 64, None, 0, None, None, None, None, 0,
                             None) == 0
    assert lib.mosaic_sample_signs(ctypes.byref(r), 0, None, None) == 0
    assert lib.mosaic_hadamard_rotate(None, 64, None, 64, 0, 64, 64, None, 0, None) == 0
    assert lib.mosaic_quantize_rows(None, 8, 0, 8, 127, None, 0, None, 0, None, None) == 0
