"""The check against a regenerated reference (krex_check_gen) vs the oracle's
generation of that reference followed by its check, field by field at 0 ULP:
all 16 dtype pairs, uniform (power-of-two and other ranges), normal and
bitcast references, ragged sizes, word offsets that are multiples of 4 (the
vector path) and ones that are not, a misaligned candidate, n = 0; then
equality with the two-operand GPU check at 2^24 + 7 elements and on the
check-stress command's full 268,435,456 fp16 elements, and exact records at
the largest n, 2^33 - 1."""
import pytest
import torch

import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import TORCH_DT, empty, from_storage, same_result

pytestmark = pytest.mark.gpu

DTS = ["f32", "bf16", "f16", "f8"]
DISTS = [(0, -4.0, 4.0), (0, 0.1, 0.7), (1, 0.0, 1.0), (2, 0.0, 0.0)]
TOL = {"f32": (1e-4, 1e-5), "bf16": (1.6e-2, 1e-2), "f16": (1e-3, 1e-3), "f8": (0.125, 0.125)}
SIZES = [1, 3, 17, 4099, 65541]
OFFSETS = [0, 4, 1, 3, 4 * (2**33) + 6]


def _candidate(dta, dtb, n, seed, off, d, p0, p1):
    """The reference's own stream generated in dta (values equal up to
    rounding), then 2% of elements perturbed (ROUND mode, delta 0.05)."""
    a = oracle.gen(dta, n, seed, off, d, p0, p1)
    a, _ = oracle.inject(a, dta, seed + 7, 0.02, 0.05, oracle.INJ_ROUND)
    return a


def _one(dta, dtb, n, seed, off, d, p0, p1, misalign=False):
    a = _candidate(dta, dtb, n, seed, off, d, p0, p1)
    b = oracle.gen(dtb, n, seed, off, d, p0, p1)
    rtol, atol = TOL[dtb]
    ref = oracle.check(a, dta, b, dtb, rtol, atol)
    ga = from_storage(a, dta)
    if misalign:                     # element-aligned, not 16-byte aligned
        buf = empty(dta, n + 1)
        buf[1:].copy_(ga)
        ga = buf[1:]
    r = krex.check_gen(ga, TORCH_DT[dtb], seed, rtol, atol, offset=off, dist=d, p0=p0, p1=p1)
    same_result(r, ref)


@pytest.mark.parametrize("dta", DTS)
@pytest.mark.parametrize("dtb", DTS)
@pytest.mark.parametrize("dist", DISTS, ids=lambda d: "%d_%g_%g" % d)
def test_check_gen_matches_oracle(dta, dtb, dist):
    d, p0, p1 = dist
    for n in SIZES:
        for off in OFFSETS:
            _one(dta, dtb, n, 31, off, d, p0, p1)
    _one(dta, dtb, 65541, 32, 8, d, p0, p1, misalign=True)
    _one(dta, dtb, (1 << 20) + 5, 33, 0, d, p0, p1)
    _one(dta, dtb, (1 << 20) + 5, 34, 2, d, p0, p1)


def test_check_gen_empty_and_exact():
    out = krex.check_gen(empty("f16", 0), torch.float16, 1, 0.0, 0.0)
    assert out.n == 0 and out.mismatches == 0 and out.argmax_abs == 2**64 - 1
    # a candidate equal to the reference: no mismatch, every maximum 0
    x = empty("bf16", 100003)
    krex.gen(x, 9, 12, "normal", 0.5, 2.0)
    r = krex.check_gen(x, torch.bfloat16, 9, 0.0, 0.0, offset=12, dist="normal", p0=0.5, p1=2.0)
    assert (r.mismatches, r.nan_count, r.max_abs, r.max_rel) == (0, 0, 0.0, 0.0)
    assert r.argmax_abs == 0


@pytest.mark.parametrize("pair", [("f32", "f32"), ("bf16", "f32"), ("f16", "f16"), ("f8", "f8"), ("f32", "f8"),
                                  ("f8", "bf16")], ids=lambda p: "%sx%s" % p)
def test_check_gen_equals_two_operand_check(pair):
    """On the GPU at 2^24 + 7 elements: the record equals krex_check's with
    the reference generated into memory."""
    dta, dtb = pair
    n = (1 << 24) + 7
    for d, p0, p1 in DISTS:
        for off in (0, 5):
            a = empty(dta, n)
            krex.gen(a, 41, off, d, p0, p1)
            krex.inject(a, a, 42, 0.001, 0.25, "round")
            b = empty(dtb, n)
            krex.gen(b, 41, off, d, p0, p1)
            rtol, atol = TOL[dtb]
            r1 = krex.check(a, b, rtol, atol)
            r2 = krex.check_gen(a, b.dtype, 41, rtol, atol, offset=off, dist=d, p0=p0, p1=p1)
            assert r1 == r2, (pair, d, off, r1, r2)


def test_check_stress_with_the_regenerated_reference():
    """The check-stress command (268,435,456 fp16 elements): checking y
    against x regenerated gives the two-operand check's record."""
    from paper_2609_30057_amd import workloads as W
    cfg = W.CHECK_STRESS
    m = cfg["rows"] * cfg["cols"]
    x = torch.empty(m, dtype=torch.float16, device="cuda")
    y = torch.empty_like(x)
    krex.gen_inject(x, y, cfg["seed"], 0, "uniform", cfg["p0"], cfg["p1"], mask_seed=cfg["mask_seed"],
                    rate=cfg["rate"], delta=cfg["delta"], mode="exact")
    r1 = krex.check(y, x, cfg["rtol"], cfg["atol"])
    del x
    r2 = krex.check_gen(y, torch.float16, cfg["seed"], cfg["rtol"], cfg["atol"], dist="uniform", p0=cfg["p0"],
                        p1=cfg["p1"])
    assert r1 == r2
    assert r2.max_abs == 0.5 and r2.nan_count == 0 and r2.mismatches > 250000


def test_check_gen_rejects_bad_arguments():
    a = empty("f16", 64)
    for kw in (dict(dist="uniform", p0=1.0, p1=-1.0), dict(dist="normal", p0=0.0, p1=-1.0)):
        with pytest.raises(krex.KrexError) as e:
            krex.check_gen(a, torch.float16, 1, 0.0, 0.0, **kw)
        assert e.value.status == krex.EINVAL
    with pytest.raises(krex.KrexError):
        krex.check_gen(a, torch.float16, 1, -1.0, 0.0)
    with pytest.raises(krex.KrexError):
        krex.check_gen(a, torch.int32, 1, 0.0, 0.0)
    with pytest.raises(krex.KrexError):
        krex.check_gen(a, torch.float16, 1, 0.0, 0.0, offset=2**64 - 8)


def _plant(a, idx, byte):
    """Sets fp8 element i of a to the bit pattern `byte`; returns the
    values before and after (exact fp32)."""
    v = a.view(torch.uint8)
    before = [float(a[i].float().item()) for i in idx]
    for i in idx:
        v[i] = byte
    after = [float(a[i].float().item()) for i in idx]
    return before, after


def test_check_gen_at_the_largest_n():
    """n = 2^33 - 1 fp8 elements against the regenerated reference: zero
    record for the generated tensor itself, then three planted changes on
    both sides of index 2^32 and in the n mod 16 tail give the exact
    record."""
    n = 2**33 - 1
    a = torch.empty(n, dtype=torch.float8_e4m3fn, device="cuda")
    krex.gen(a, 71, 0, "uniform", -4.0, 4.0)
    r = krex.check_gen(a, torch.float8_e4m3fn, 71, 0.0, 0.0, dist="uniform", p0=-4.0, p1=4.0)
    assert (r.n, r.mismatches, r.nan_count, r.max_abs, r.argmax_abs, r.max_rel) == (n, 0, 0, 0.0, 0, 0.0)
    idx = [5, 2**32 + 9, n - 1]
    before, after = _plant(a, idx, 0x58)              # 0x58 = 16.0, outside [-4, 4]
    r = krex.check_gen(a, torch.float8_e4m3fn, 71, 0.0, 0.0, dist="uniform", p0=-4.0, p1=4.0)
    d = [abs(x - y) for x, y in zip(after, before)]
    assert r.mismatches == 3 and r.nan_count == 0
    assert r.max_abs == max(d) and r.argmax_abs == idx[d.index(max(d))]
    del a
    torch.cuda.empty_cache()
