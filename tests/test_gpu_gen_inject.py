"""Generation and injection in one call (krex_gen_inject) vs the oracle's
generation followed by its injection, bit for bit, and vs the two separate
GPU calls: every dtype, uniform (power-of-two and other ranges), normal and
bitcast values, both injection modes, ragged sizes, offsets that are
multiples of 4 (the fused kernel) and ones that are not (the two kernels in
order), and the check-stress command at its full size."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import assert_bits_equal, empty, to_storage

pytestmark = pytest.mark.gpu

DTS = ["f32", "bf16", "f16", "f8"]
DISTS = [(0, -4.0, 4.0), (0, 0.1, 0.7), (1, 0.0, 1.0), (2, 0.0, 0.0)]
SIZES = [1, 3, 17, 4099, (1 << 20) + 5]
OFFSETS = [(0, 0), (4, 8), (65536, 0), (4 * (2**32 - 1) - 8, 12), (1, 3)]   # (value, mask); the last: unaligned


def _ref(dt, n, seed, off, d, p0, p1, mseed, moff, rate, delta, mode):
    x = oracle.gen(dt, n, seed, off, d, p0, p1)
    y, _ = oracle.inject(x, dt, mseed, rate, delta, mode, moff)
    return x, y


@pytest.mark.parametrize("dt", DTS)
@pytest.mark.parametrize("dist", DISTS, ids=lambda d: "%d_%g_%g" % d)
def test_gen_inject_matches_oracle(dt, dist):
    d, p0, p1 = dist
    for mode, delta in (("exact", 0.5), ("round", 1.0)):
        m = oracle.INJ_EXACT if mode == "exact" else oracle.INJ_ROUND
        for n in SIZES:
            for off, moff in OFFSETS:
                x, y = empty(dt, n), empty(dt, n)
                krex.gen_inject(x, y, 21, off, d, p0, p1, mask_seed=22, rate=0.05, delta=delta, mode=mode,
                                mask_offset=moff)
                xr, yr = _ref(dt, n, 21, off, d, p0, p1, 22, moff, 0.05, delta, m)
                what = "%s dist=%s %s n=%d off=%d moff=%d" % (dt, dist, mode, n, off, moff)
                assert_bits_equal(to_storage(x, dt), xr, what + " x")
                assert_bits_equal(to_storage(y, dt), yr, what + " y")


@pytest.mark.parametrize("dt", DTS)
def test_gen_inject_equals_separate_calls(dt):
    """Large tensors, rate 1 (every element perturbed) and rate 0 too."""
    n = (1 << 24) + 7
    for d, p0, p1 in ((0, -1.0, 1.0), (1, 0.0, 1.0)):
        for rate in (0.001, 1.0, 0.0):
            x, y = empty(dt, n), empty(dt, n)
            krex.gen_inject(x, y, 5, 0, d, p0, p1, mask_seed=6, rate=rate, delta=0.25, mode="exact")
            xs, ys = empty(dt, n), empty(dt, n)
            krex.gen(xs, 5, 0, d, p0, p1)
            krex.inject(ys, xs, 6, rate, 0.25, "exact")
            assert torch.equal(x.view(torch.uint8), xs.view(torch.uint8)), (dt, d, rate)
            assert torch.equal(y.view(torch.uint8), ys.view(torch.uint8)), (dt, d, rate)


def test_check_stress_through_the_fused_call():
    """The check-stress command's x and y (268,435,456 fp16) from one call
    equal the separate calls; the check's closed forms hold."""
    from paper_2609_30057_amd import workloads as W
    cfg = W.CHECK_STRESS
    m = cfg["rows"] * cfg["cols"]
    x = torch.empty(m, dtype=torch.float16, device="cuda")
    y = torch.empty_like(x)
    krex.gen_inject(x, y, cfg["seed"], 0, "uniform", cfg["p0"], cfg["p1"], mask_seed=cfg["mask_seed"],
                    rate=cfg["rate"], delta=cfg["delta"], mode="exact")
    r = krex.check(y, x, cfg["rtol"], cfg["atol"])
    xs = torch.empty_like(x)
    krex.gen(xs, cfg["seed"], 0, "uniform", cfg["p0"], cfg["p1"])
    assert torch.equal(x.view(torch.int16), xs.view(torch.int16))
    ys = torch.empty_like(x)
    krex.inject(ys, xs, cfg["mask_seed"], cfg["rate"], cfg["delta"], "exact")
    assert torch.equal(y.view(torch.int16), ys.view(torch.int16))
    del xs, ys
    assert r.max_abs == 0.5 and r.nan_count == 0
    changed = int((x.view(torch.int16) != y.view(torch.int16)).sum().item())
    assert r.mismatches == changed
    first = int(torch.nonzero(x.view(torch.int16) != y.view(torch.int16))[0].item())
    assert r.argmax_abs == first


def test_gen_inject_rejects_bad_arguments():
    x = empty("f16", 64)
    with pytest.raises(krex.KrexError) as e:
        krex.gen_inject(x, x, 1, rate=0.1, delta=0.5)              # outputs overlap
    assert e.value.status == krex.EINVAL
    buf = empty("f16", 100)
    with pytest.raises(krex.KrexError):
        krex.gen_inject(buf[:64], buf[32:96], 1, rate=0.1, delta=0.5)
    w = torch.empty(64, dtype=torch.int32, device="cuda")
    with pytest.raises(krex.KrexError):
        krex.gen_inject(w, torch.empty_like(w), 1, rate=0.1, delta=0.5)   # raw words cannot be perturbed
    with pytest.raises(krex.KrexError):
        krex.gen_inject(x, empty("f16", 64), 1, rate=1.5, delta=0.5)
    with pytest.raises(krex.KrexError):
        krex.gen_inject(x, empty("f16", 64), 1, dist="uniform", p0=1.0, p1=-1.0, rate=0.1, delta=0.5)
    y = empty("f16", 0)
    krex.gen_inject(empty("f16", 0), y, 1, rate=0.1, delta=0.5)          # n = 0: nothing to do
