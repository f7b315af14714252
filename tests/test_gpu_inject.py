"""GPU mismatch injection vs the oracle, bit for bit, for every dtype, both
modes, rates 0 / small / large / 1, signed deltas, mask offsets (aligned and
not), in place and out of place, ragged sizes."""
import numpy as np
import pytest

import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import assert_bits_equal, empty, from_storage, to_storage

pytestmark = pytest.mark.gpu

DTS = ["f32", "bf16", "f16", "f8"]


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("mode", ["round", "exact"])
def test_inject_matches_oracle(dt, mode):
    m = {"round": 0, "exact": 1}[mode]
    for n in (0, 1, 7, 33, 10007, (1 << 20) + 3):
        x_ref = oracle.gen(dt, n, 5, 0, 0, -4.0, 4.0)
        for rate, delta, moff in ((0.0, 0.5, 0), (0.001, 0.5, 0), (0.3, -0.25, 3), (1.0, 1.0, 65536),
                                  (0.05, 0.5, 1)):
            y_ref, _ = oracle.inject(x_ref, dt, 6, rate, delta, m, moff)
            x = from_storage(x_ref, dt)
            y = empty(dt, n)
            krex.inject(y, x, 6, rate, delta, mode, moff)
            what = "%s %s n=%d rate=%g delta=%g moff=%d" % (dt, mode, n, rate, delta, moff)
            assert_bits_equal(to_storage(y, dt), y_ref, what)
            krex.inject(x, x, 6, rate, delta, mode, moff)          # in place
            assert_bits_equal(to_storage(x, dt), y_ref, what + " in place")


def test_inject_special_inputs():
    """NaN, infinities and signed zeros in x pass through both modes exactly as
    the oracle decides."""
    bits = oracle.words(50000, 8, 0)
    x_ref = bits.view(np.float32).copy()
    for dt in DTS:
        xs = oracle.from_f32(x_ref, dt) if dt != "f32" else x_ref
        for m, mode in ((0, "round"), (1, "exact")):
            y_ref, _ = oracle.inject(xs, dt, 9, 0.5, 0.75, m)
            x = from_storage(xs, dt)
            y = empty(dt, xs.size)
            krex.inject(y, x, 9, 0.5, 0.75, mode)
            assert_bits_equal(to_storage(y, dt), y_ref, "%s %s specials" % (dt, mode))


def test_inject_rejects_partial_overlap():
    buf = empty("f16", 1024)
    with pytest.raises(krex.KrexError):
        krex.inject(buf[8:520], buf[0:512], 1, 0.1, 0.5)
    with pytest.raises(krex.KrexError):
        krex.inject(buf[:16], buf[16:32], 1, 1.5, 0.5)
