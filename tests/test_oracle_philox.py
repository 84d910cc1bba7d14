"""Pins for the oracle's Philox generator (CPU only)."""
import os
import shutil
import subprocess
from decimal import Decimal, getcontext

import numpy as np
import pytest

from oracle.philox import PHILOX_CONSTANTS, philox4x32_np, philox_generic
from oracle.sampling import stream_words


def _numpy_philox_block(ctr, key):
    """numpy.random.Philox (Philox-4x64-10) output for counter ``ctr``.
    numpy increments the counter before producing a block, so the state is
    set one below the wanted counter."""
    bg = np.random.Philox()
    st = bg.state
    c = list(ctr)
    c[0] = (c[0] - 1) % (1 << 64)
    borrow = ctr[0] == 0
    for w in range(1, 4):
        if not borrow:
            break
        borrow = c[w] == 0
        c[w] = (c[w] - 1) % (1 << 64)
    st["state"]["counter"] = np.array(c, dtype=np.uint64)
    st["state"]["key"] = np.array(key, dtype=np.uint64)
    st["buffer_pos"] = 4
    bg.state = st
    return tuple(int(v) for v in bg.random_raw(4))


@pytest.mark.parametrize("ctr,key", [
    ((5, 7, 11, 13), (0x0123456789ABCDEF, 0xFEDCBA9876543210)),
    ((0, 0, 0, 0), (0, 0)),
    ((2 ** 64 - 1, 2 ** 64 - 1, 2 ** 64 - 1, 2 ** 64 - 1), (2 ** 64 - 1, 2 ** 64 - 1)),
    ((1, 0, 0, 0), (1, 0)),
    ((0x243F6A8885A308D3, 0x13198A2E03707344, 0xA4093822299F31D0, 0x082EFA98EC4E6C89),
     (0x452821E638D01377, 0xBE5466CF34E90C6C)),
])
def test_generic_philox_4x64_matches_numpy(ctr, key):
    assert philox_generic(ctr, key, width=64) == _numpy_philox_block(ctr, key)


def test_generic_philox_4x64_random_against_numpy():
    rng = np.random.default_rng(123)
    for _ in range(50):
        ctr = tuple(int(v) for v in rng.integers(0, 2 ** 64, 4, dtype=np.uint64, endpoint=False))
        key = tuple(int(v) for v in rng.integers(0, 2 ** 64, 2, dtype=np.uint64, endpoint=False))
        assert philox_generic(ctr, key, width=64) == _numpy_philox_block(ctr, key)


def test_weyl_constants_closed_form():
    """The key increments are the fractional parts of the golden ratio and
    of sqrt(3), scaled to W bits."""
    getcontext().prec = 80
    phi_frac = (Decimal(5).sqrt() - 1) / 2
    s3_frac = Decimal(3).sqrt() - 1
    for w in (32, 64):
        w0, w1 = PHILOX_CONSTANTS[w]["W"]
        assert w0 == int(phi_frac * (2 ** w))
        assert w1 == int(s3_frac * (2 ** w))


ROCRAND_HEADER = "/opt/rocm/include/rocrand/rocrand_philox4x32_10.h"


@pytest.fixture(scope="module")
def rocrand_block(tmp_path_factory):
    """rocRAND's Philox-4x32-10 block function, built on the host from its
    open-source header (an implementation independent of the oracle)."""
    if not os.path.exists(ROCRAND_HEADER) or shutil.which("g++") is None:
        pytest.skip("rocRAND header or g++ not available")
    exe = str(tmp_path_factory.mktemp("rocrand") / "philox_ref")
    src = os.path.join(os.path.dirname(__file__), "rocrand_philox_ref.cpp")
    subprocess.run(["g++", "-O1", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", src, "-o", exe],
                   check=True, capture_output=True)

    def run(pairs):
        text = "".join(" ".join(str(int(v)) for v in (*c, *k)) + "\n" for c, k in pairs)
        out = subprocess.run([exe], input=text, capture_output=True, text=True, check=True).stdout
        return [tuple(int(v) for v in line.split()) for line in out.strip().splitlines()]
    return run


def test_philox4x32_matches_rocrand(rocrand_block):
    """The 4x32 instance (multipliers 0xD2511F53 / 0xCD9E8D57, ten rounds)
    equals rocRAND's Philox4x32-10 on 64 random (counter, key) pairs and on
    all-zero, all-one and digits-of-pi inputs; a wrong multiplier, Weyl
    increment, round count or output permutation fails it."""
    m = 2 ** 32 - 1
    pairs = [((0, 0, 0, 0), (0, 0)), ((m, m, m, m), (m, m)),
             ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0)),
             ((1, 0, 0, 0), (0, 0)), ((0, 0, 0, 1), (0, 1))]
    rng = np.random.default_rng(2024)
    for _ in range(64):
        c = tuple(int(v) for v in rng.integers(0, 2 ** 32, 4, dtype=np.uint64))
        k = tuple(int(v) for v in rng.integers(0, 2 ** 32, 2, dtype=np.uint64))
        pairs.append((c, k))
    ref = rocrand_block(pairs)
    assert len(ref) == len(pairs)
    for (c, k), r in zip(pairs, ref):
        assert philox_generic(c, k, width=32) == r
    c = np.array([p[0] for p in pairs], dtype=np.uint64).T
    for (c_, k), r in zip(pairs, ref):
        out = philox4x32_np(*[np.array([v], dtype=np.uint64) for v in c_], k[0], k[1])
        assert tuple(int(o[0]) for o in out) == r


def test_stream_words_match_rocrand(rocrand_block):
    """The oracle's stream (key = seed halves, counter = (block lo, block hi,
    stream, instance)) built on rocRAND's block function."""
    seed, st, inst = 0x0123_4567_89AB_CDEF, 0x51, 7
    words = stream_words(seed, st, inst, 0, 64)
    pairs = [((b, 0, st, inst), (seed & 0xFFFFFFFF, seed >> 32)) for b in range(16)]
    ref = rocrand_block(pairs)
    assert [int(w) for w in words] == [v for blk in ref for v in blk]


def test_multipliers_odd():
    for w in (32, 64):
        for m in PHILOX_CONSTANTS[w]["M"]:
            assert m % 2 == 1 and m < 2 ** w


def test_vectorised_4x32_matches_generic():
    rng = np.random.default_rng(7)
    c = rng.integers(0, 2 ** 32, (4, 200), dtype=np.uint64)
    k = [int(v) for v in rng.integers(0, 2 ** 32, 2, dtype=np.uint64)]
    out = philox4x32_np(c[0], c[1], c[2], c[3], k[0], k[1])
    for i in range(200):
        ref = philox_generic([int(c[j, i]) for j in range(4)], k, width=32)
        assert tuple(int(out[j][i]) for j in range(4)) == ref


def test_rounds_matter():
    """Fewer rounds give a different function (guards a loop that stops early)."""
    a = philox_generic((1, 2, 3, 4), (5, 6), 32, 10)
    b = philox_generic((1, 2, 3, 4), (5, 6), 32, 9)
    assert a != b


def test_stream_words_mapping():
    """Word t of stream (seed, s, inst) is word t mod 4 of the block t div 4,
    including offsets that are not multiples of 4 and block indices >= 2^32."""
    seed = 0x1234_5678_9ABC_DEF0
    words = stream_words(seed, 0x51, 9, 5, 11)
    for i in range(11):
        t = 5 + i
        b = t // 4
        ref = philox_generic((b & 0xFFFFFFFF, b >> 32, 0x51, 9),
                             (seed & 0xFFFFFFFF, seed >> 32), 32)
        assert int(words[i]) == ref[t % 4]
    t0 = 4 * (2 ** 32) + 2
    w = stream_words(seed, 3, 4, t0, 3)
    for i in range(3):
        t = t0 + i
        b = t // 4
        ref = philox_generic((b & 0xFFFFFFFF, b >> 32, 3, 4), (seed & 0xFFFFFFFF, seed >> 32), 32)
        assert int(w[i]) == ref[t % 4]


def test_words_look_uniform():
    w = stream_words(99, 1, 0, 0, 1 << 20)
    by = np.frombuffer(w.tobytes(), dtype=np.uint8)
    counts = np.bincount(by, minlength=256)
    exp = by.size / 256
    chi2 = float(((counts - exp) ** 2 / exp).sum())
    assert chi2 < 400  # 255 dof: mean 255, sd ~22.6
    bits = np.unpackbits(by)
    assert abs(bits.mean() - 0.5) < 2e-3


def test_c_stream_generator_matches_definition():
    """The oracle's C generator (used for long ranges) equals the numpy one
    and the scalar definition, including block-unaligned starts and counters
    past 2^32 blocks."""
    from oracle import _cstream
    from oracle.sampling import stream_words_np
    for seed, st, inst, t0, n in [(0x1234_5678_9ABC_DEF0, 0x51, 9, 5, 5000), (7, 0x20, 0, 0, 4096),
                                  (2 ** 64 - 1, 3, 2 ** 32 - 1, 4 * (2 ** 32) - 6, 4100)]:
        c = _cstream.stream_words(seed, st, inst, t0, n)
        assert np.array_equal(c, stream_words_np(seed, st, inst, t0, n))
        for i in (0, 1, n // 2, n - 1):
            t = t0 + i
            ref = philox_generic(((t // 4) & 0xFFFFFFFF, (t // 4) >> 32, st, inst),
                                 (seed & 0xFFFFFFFF, seed >> 32), 32)
            assert int(c[i]) == ref[t % 4]
