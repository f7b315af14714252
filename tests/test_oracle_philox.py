"""Pins the oracle's Philox4x32-10 word stream to two independent published
implementations (rocRAND's engine header and ATen's CPU engine header, built
on the host by tests/pins) and to a third, pure-Python transcription of the
SC'11 round function used only on a handful of blocks.

The stream is the seeded-generation reading of Section 2.1 ("Benchmarking
command": generation must not depend on colocated work), realised as a
counter-based generator so that every element's word is a pure function of
(seed, offset + j)."""
import numpy as np
import pytest

from tests.pins import build as pins

SEEDS = [0, 1, 2, 3, 4, 0xFFFFFFFF, 0x100000000, 0xDEADBEEFCAFEF00D, 2**64 - 1]


@pytest.fixture(scope="module")
def xc():
    return pins.load()


@pytest.mark.parametrize("seed", SEEDS)
def test_first_million_words_match_rocrand_and_aten(oracle_mod, xc, seed):
    n = 1 << 20
    ours = oracle_mod.words(n, seed, 0)
    assert np.array_equal(ours, pins.rocrand_words(xc, seed, 0, n))
    assert np.array_equal(ours, pins.aten_words(xc, seed, 0, n))


@pytest.mark.parametrize("offset", [1, 2, 3, 5, 65536, 16777216, 268435455, 2**40 + 3])
def test_offsets_match(oracle_mod, xc, offset):
    n = 4099
    for seed in (0, 2, 2**64 - 1):
        ours = oracle_mod.words(n, seed, offset)
        assert np.array_equal(ours, pins.rocrand_words(xc, seed, offset, n))
        assert np.array_equal(ours, pins.aten_words(xc, seed, offset, n))


def test_block_counter_carry(oracle_mod, xc):
    """Block index b = 2^32 - 1 -> 2^32 carries into the second counter word."""
    off = 4 * (2**32 - 1) - 6
    n = 32
    for seed in (0, 7):
        ours = oracle_mod.words(n, seed, off)
        assert np.array_equal(ours, pins.rocrand_words(xc, seed, off, n))
        assert np.array_equal(ours, pins.aten_words(xc, seed, off, n))


def test_single_word_equals_bulk(oracle_mod):
    w = oracle_mod.words(64, 5, 1000)
    for j in range(64):
        assert oracle_mod.word(5, 1000 + j) == int(w[j])


def _py_philox(ctr, key):
    """Third opinion on a few blocks: the round function and key schedule of
    Philox4x32-10 as described in SC'11, in Python integers."""
    M0, M1, W0, W1 = 0xD2511F53, 0xCD9E8D57, 0x9E3779B9, 0xBB67AE85
    x = list(ctr)
    k0, k1 = key
    mask = 0xFFFFFFFF
    for _ in range(10):
        p0 = M0 * x[0]
        p1 = M1 * x[2]
        x = [((p1 >> 32) ^ x[1] ^ k0) & mask, p1 & mask, ((p0 >> 32) ^ x[3] ^ k1) & mask, p0 & mask]
        k0 = (k0 + W0) & mask
        k1 = (k1 + W1) & mask
    return x


def test_python_transcription_agrees(oracle_mod):
    rng = np.random.default_rng(11)
    for _ in range(50):
        ctr = [int(v) for v in rng.integers(0, 2**32, 4, dtype=np.uint64)]
        key = [int(v) for v in rng.integers(0, 2**32, 2, dtype=np.uint64)]
        assert oracle_mod.philox(ctr, key) == _py_philox(ctr, key)


def test_words_look_uniform(oracle_mod):
    """Sanity on the stream statistics: byte histogram and mean of 2^22 words."""
    w = oracle_mod.words(1 << 22, 123, 0)
    mean = w.astype(np.float64).mean() / 2**32
    assert abs(mean - 0.5) < 5 * (1 / np.sqrt(12 * w.size))
    hist = np.bincount((w & 0xFF).astype(np.int64), minlength=256)
    exp = w.size / 256
    chi2 = ((hist - exp) ** 2 / exp).sum()
    assert chi2 < 400  # 255 dof; p < 1e-6 above ~370
