"""GPU generation vs the oracle, bit for bit: every dtype and distribution,
ragged and tiny sizes, unaligned offsets (including the 32-bit block-counter
carry), extreme seeds and misaligned destination pointers; the value
transforms over every possible input through krex_transform_words."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import assert_bits_equal, empty, from_storage, to_storage

pytestmark = pytest.mark.gpu

DTS = ["f32", "bf16", "f16", "f8"]
# Uniform ranges: powers of two (-1..1, -4..4, 1000..1016: one fused
# multiply-add in the kernel), 2^-110 (a power of two whose 2^-24 step would
# be subnormal) and 0.6 take the two-rounding path.
DISTS = [(0, -1.0, 1.0), (0, -4.0, 4.0), (0, 0.1, 0.7), (1, 0.0, 1.0), (1, 2.5, 0.5), (2, 0.0, 0.0),
         (0, 1000.0, 1016.0), (0, 0.0, 2.0**-110)]
SIZES = [0, 1, 3, 15, 17, 4099, (1 << 20) + 5]
OFFSETS = [0, 1, 3, 65536, 4 * (2**32 - 1) - 6]
SEEDS = [0, 2**64 - 1]


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("dist", DISTS, ids=lambda d: "%d_%g_%g" % d)
def test_gen_matches_oracle(dt, dist):
    d, p0, p1 = dist
    for n in SIZES:
        for off in OFFSETS:
            for seed in SEEDS:
                t = empty(dt, n)
                krex.gen(t, seed, off, d, p0, p1)
                ref = oracle.gen(dt, n, seed, off, d, p0, p1)
                assert_bits_equal(to_storage(t, dt), ref, "%s dist=%s n=%d off=%d seed=%d" % (dt, dist, n, off, seed))


def test_raw_words_match_oracle():
    for n in SIZES:
        for off in OFFSETS:
            t = empty("u32", n)
            krex.gen(t, 12345, off)
            assert_bits_equal(to_storage(t, "u32"), oracle.words(n, 12345, off), "u32 n=%d off=%d" % (n, off))


@pytest.mark.parametrize("dt", DTS + ["u32"])
def test_misaligned_destination(dt):
    """dst one element past a 16-byte boundary takes the element-wise path."""
    n = 10007
    for d, p0, p1 in DISTS[:1] + DISTS[3:4]:
        buf = empty(dt, n + 1)
        t = buf[1:]
        krex.gen(t, 77, 4, d, p0, p1)
        ref = oracle.gen(dt, n, 77, 4, d, p0, p1)
        assert_bits_equal(to_storage(t, dt), ref, "%s misaligned" % dt)


@pytest.mark.parametrize("dt", DTS)
def test_large_gen(dt):
    n = (1 << 24) + 3
    for d, p0, p1 in (DISTS[1], DISTS[3]):
        t = empty(dt, n)
        krex.gen(t, 2, 0, d, p0, p1)
        assert_bits_equal(to_storage(t, dt), oracle.gen(dt, n, 2, 0, d, p0, p1), "%s large" % dt)


def test_normal_transform_every_u1_and_angle():
    """rho over all 2^24 values of u1 (angle 0) and the angle over all 2^24
    values (u1 fixed), through krex_transform_words, equal the oracle."""
    k = np.arange(1 << 24, dtype=np.uint32)
    for w in (np.stack([k << 8, np.zeros_like(k)], 1).reshape(-1),
              np.stack([np.full_like(k, 0x12345600), k << 8], 1).reshape(-1),
              np.stack([k << 8 | 0xFF, (k * 2654435761) & 0xFFFFFFFF], 1).reshape(-1).astype(np.uint32)):
        words = from_storage(w, "u32")
        t = empty("f32", w.size)
        krex.transform_words(t, words, "normal", 0.0, 1.0)
        assert_bits_equal(to_storage(t, "f32"), oracle.transform_words("f32", w, 1, 0.0, 1.0), "normal words")


@pytest.mark.parametrize("dt", ["bf16", "f16", "f8"])
def test_narrowing_over_bit_patterns(dt):
    """Every 251st fp32 bit pattern, plus every pattern in the two-exponent
    windows where the format's rounding rules change (underflow to zero,
    subnormal / normal, overflow, inf / NaN), narrowed on the GPU (bitcast
    transform) and by the oracle."""
    windows = {"bf16": [(0, 2), (253, 256)], "f16": [(102, 104), (112, 114), (142, 144), (254, 256)],
               "f8": [(116, 118), (120, 122), (134, 136), (254, 256)]}[dt]
    chunks = [np.arange(s, min(s + (1 << 24) * 251, 1 << 32), 251, dtype=np.uint64).astype(np.uint32)
              for s in range(0, 1 << 32, (1 << 24) * 251)]
    for e0, e1 in windows:
        for sign in (0, 1):
            chunks.append(np.arange((sign << 31) | (e0 << 23), (sign << 31) | (e1 << 23), dtype=np.uint64)
                          .astype(np.uint32))
    for bits in chunks:
        words = from_storage(bits, "u32")
        t = empty(dt, bits.size)
        krex.transform_words(t, words, "bitcast")
        ref = oracle.from_f32(bits.view(np.float32), dt)
        assert_bits_equal(to_storage(t, dt), ref, "%s narrowing" % dt)


def test_uniform_transform_all_24bit_values():
    k = np.arange(1 << 24, dtype=np.uint32) << 8
    words = from_storage(k, "u32")
    for dt in DTS:
        for lo, hi in ((-1.0, 1.0), (0.1, 0.7), (-4.0, 4.0), (1000.0, 1016.0)):
            t = empty(dt, k.size)
            krex.transform_words(t, words, "uniform", lo, hi)
            assert_bits_equal(to_storage(t, dt), oracle.transform_words(dt, k, 0, lo, hi), "%s uniform" % dt)


def test_gen_is_launch_independent():
    """The same elements generated as one call or as pieces at their offsets
    are identical (counter-based stream)."""
    n = 1 << 20
    whole = empty("bf16", n)
    krex.gen(whole, 9, 0, "normal")
    parts = empty("bf16", n)
    cut = [0, 5, 4096, 77777, 500001, n]
    for a, b in zip(cut[:-1], cut[1:]):
        krex.gen(parts[a:b], 9, a, "normal")
    assert torch.equal(whole.view(torch.int16), parts.view(torch.int16))


def test_gen_rejects_bad_arguments():
    t = empty("f32", 16)
    with pytest.raises(krex.KrexError) as e:
        krex.gen(t, 0, 0, "uniform", 1.0, -1.0)
    assert e.value.status == krex.EINVAL
    with pytest.raises(krex.KrexError):
        krex.gen(t, 0, 2**64 - 3)
    with pytest.raises(krex.KrexError):
        krex.gen(t, 0, 0, "normal", 0.0, -1.0)


def test_gen_beyond_2_to_32_elements():
    """4 GiB of fp8 in one launch (n > 2^32) at an offset near the top of the
    word stream: elements on both sides of index 2^32 match the oracle."""
    n = 2**32 + 7
    off = 2**64 - n - 3
    t = empty("f8", n)
    krex.gen(t, 11, off, 0, -1.0, 1.0)
    idx = np.array([0, 1, 2**31, 2**32 - 1, 2**32, 2**32 + 1, n - 1])
    got = to_storage(t[torch.from_numpy(idx).cuda()], "f8")
    ref = np.concatenate([oracle.gen("f8", 1, 11, off + int(i), 0, -1.0, 1.0) for i in idx])
    assert_bits_equal(got, ref, "f8 > 2^32")
    del t
