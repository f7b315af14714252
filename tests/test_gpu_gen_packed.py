"""GPU packed-stream generation (narrow dtypes, 16 or 8 bits of the Philox
word stream per element) vs the oracle, bit for bit: every narrow dtype and
distribution, ragged and tiny sizes, field offsets that are not multiples of
the 16-byte unit (including the 32-bit block-counter carry), misaligned
destinations, a large tensor, and samples of the 268M-element shape; plus the
device-side identity that the bitcast form is the byte view of the plain
word stream."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import assert_bits_equal, empty, to_storage

pytestmark = pytest.mark.gpu

DTS = ["bf16", "f16", "f8"]
# (0, 0, 1e-37): a range whose 2^-W multiple is not exact, so the kernel's
# unscaled uniform path runs.
DISTS = [(0, -1.0, 1.0), (0, -4.0, 4.0), (0, 0.1, 0.7), (0, 0.0, 1e-37), (1, 0.0, 1.0), (1, 2.5, 0.5),
         (2, 0.0, 0.0)]
SIZES = [0, 1, 3, 15, 17, 4099, (1 << 20) + 5]


def offsets(dt, d):
    fields_per_block = 4 * 32 // oracle.packed_width(dt, d)
    return [0, 1, 3, 8, 16, 65536, fields_per_block * (2**32 - 1) - 6]


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("dist", DISTS, ids=lambda d: "%d_%g_%g" % d)
def test_gen_packed_matches_oracle(dt, dist):
    d, p0, p1 = dist
    for n in SIZES:
        for off in offsets(dt, d):
            for seed in (0, 2**64 - 1):
                t = empty(dt, n)
                krex.gen_packed(t, seed, off, d, p0, p1)
                ref = oracle.gen_packed(dt, n, seed, off, d, p0, p1)
                assert_bits_equal(to_storage(t, dt), ref, "%s dist=%s n=%d off=%d seed=%d" % (dt, dist, n, off, seed))


@pytest.mark.parametrize("dt", DTS)
def test_misaligned_destination(dt):
    n = 10007
    for d, p0, p1 in (DISTS[0], DISTS[4], DISTS[6]):
        buf = empty(dt, n + 1)
        t = buf[1:]
        krex.gen_packed(t, 77, 16, d, p0, p1)
        assert_bits_equal(to_storage(t, dt), oracle.gen_packed(dt, n, 77, 16, d, p0, p1), "%s misaligned" % dt)


@pytest.mark.parametrize("dt", DTS)
def test_large_gen_packed(dt):
    n = (1 << 24) + 3
    for d, p0, p1 in (DISTS[1], DISTS[4]):
        t = empty(dt, n)
        krex.gen_packed(t, 2, 0, d, p0, p1)
        assert_bits_equal(to_storage(t, dt), oracle.gen_packed(dt, n, 2, 0, d, p0, p1), "%s large" % dt)


@pytest.mark.parametrize("dt,dist", [("f16", (0, -4.0, 4.0)), ("f8", (0, -4.0, 4.0)), ("bf16", (1, 0.0, 1.0))])
def test_full_size_sampled(dt, dist):
    """268M elements (the check_stress shape) in one launch; 2048 sampled
    elements against the oracle element by element."""
    d, p0, p1 = dist
    n = 1 << 28
    t = empty(dt, n)
    krex.gen_packed(t, 2, 0, d, p0, p1)
    idx = np.random.default_rng(3).integers(0, n, 2048)
    idx = np.concatenate([idx, [0, 1, n - 2, n - 1]])
    got = to_storage(t[torch.from_numpy(idx).cuda()], dt)
    ref = np.concatenate([oracle.gen_packed(dt, 1, 2, int(i), d, p0, p1) for i in idx])
    assert_bits_equal(got, ref, "%s sampled" % dt)
    del t


@pytest.mark.parametrize("dt", DTS)
def test_bitcast_is_the_word_stream_bytes(dt):
    n = 1 << 16
    t = empty(dt, n)
    krex.gen_packed(t, 99, 0, "bitcast")
    w = empty("u32", n * t.element_size() // 4)
    krex.gen(w, 99, 0)
    assert torch.equal(t.view(torch.uint8), w.view(torch.uint8))
