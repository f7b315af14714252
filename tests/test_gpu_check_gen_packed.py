"""The check against a reference regenerated from the packed stream
(krex_check_gen_packed) vs the oracle's packed generation of that reference
followed by its check, field by field at 0 ULP: every candidate dtype
against bf16, fp16 and fp8 references; uniform ranges that take each of the
three uniform modes (fused multiply-add, scaled, word transform), normal and
bitcast; ragged sizes; offsets that are multiples of a unit (the vector
path) and ones that are not (the shifted element path); a misaligned
candidate; then equality with the two-operand GPU check at 2^24 + 7
elements, and exact records at the largest n, 2^33 - 1."""
import pytest
import torch

import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import TORCH_DT, empty, from_storage, same_result

pytestmark = pytest.mark.gpu

DTA = ["f32", "bf16", "f16", "f8"]
DTB = ["bf16", "f16", "f8"]
# (dist, p0, p1): fused ([-4, 4), a power-of-two range), scaled ([0.1, 0.7)),
# word transform (a range whose 2^-W multiple is not exact), normal, bitcast
DISTS = [(0, -4.0, 4.0), (0, 0.1, 0.7), (0, 0.0, 2.0 ** -110), (1, 0.0, 1.0), (2, 0.0, 0.0)]
TOL = {"f32": (1e-4, 1e-5), "bf16": (1.6e-2, 1e-2), "f16": (1e-3, 1e-3), "f8": (0.125, 0.125)}
SIZES = [1, 3, 17, 4099, 65541]
OFFSETS = [0, 16, 1, 5, 13, 2 ** 36 + 8]


def _candidate(b, dtb, dta, seed):
    """The reference widened and rounded to dta, then 2% of it perturbed
    (ROUND mode, delta 0.05)."""
    f = oracle.to_f32(b, dtb)
    a = f if dta == "f32" else oracle.from_f32(f, dta)
    a, _ = oracle.inject(a, dta, seed + 7, 0.02, 0.05, oracle.INJ_ROUND)
    return a


def _one(dta, dtb, n, seed, off, d, p0, p1, misalign=False):
    b = oracle.gen_packed(dtb, n, seed, off, d, p0, p1)
    a = _candidate(b, dtb, dta, seed)
    rtol, atol = TOL[dtb]
    ref = oracle.check(a, dta, b, dtb, rtol, atol)
    ga = from_storage(a, dta)
    if misalign:                     # element-aligned, not 16-byte aligned
        buf = empty(dta, n + 1)
        buf[1:].copy_(ga)
        ga = buf[1:]
    r = krex.check_gen_packed(ga, TORCH_DT[dtb], seed, rtol, atol, offset=off, dist=d, p0=p0, p1=p1)
    same_result(r, ref)


@pytest.mark.parametrize("dta", DTA)
@pytest.mark.parametrize("dtb", DTB)
@pytest.mark.parametrize("dist", DISTS, ids=lambda d: "%d_%g_%g" % d)
def test_check_gen_packed_matches_oracle(dta, dtb, dist):
    d, p0, p1 = dist
    for n in SIZES:
        for off in OFFSETS:
            _one(dta, dtb, n, 51, off, d, p0, p1)
    _one(dta, dtb, 65541, 52, 32, d, p0, p1, misalign=True)
    _one(dta, dtb, (1 << 20) + 5, 53, 0, d, p0, p1)
    _one(dta, dtb, (1 << 20) + 5, 54, 7, d, p0, p1)


@pytest.mark.parametrize("pair", [("f16", "f16"), ("bf16", "bf16"), ("f8", "f8"), ("f32", "f16"), ("f8", "bf16")],
                         ids=lambda p: "%sx%s" % p)
def test_check_gen_packed_equals_two_operand_check(pair):
    """On the GPU at 2^24 + 7 elements: the record equals krex_check's with
    the packed reference generated into memory."""
    dta, dtb = pair
    n = (1 << 24) + 7
    for d, p0, p1 in DISTS:
        for off in (0, 3):
            b = empty(dtb, n)
            krex.gen_packed(b, 61, off, d, p0, p1)
            a = b.to(TORCH_DT[dta]) if dta != dtb else b.clone()
            krex.inject(a, a, 62, 0.001, 0.25, "round")
            rtol, atol = TOL[dtb]
            r1 = krex.check(a, b, rtol, atol)
            r2 = krex.check_gen_packed(a, b.dtype, 61, rtol, atol, offset=off, dist=d, p0=p0, p1=p1)
            assert r1 == r2, (pair, d, off, r1, r2)


def test_check_gen_packed_empty_and_rejections():
    out = krex.check_gen_packed(empty("f16", 0), torch.float16, 1, 0.0, 0.0)
    assert out.n == 0 and out.argmax_abs == 2**64 - 1
    a = empty("f16", 64)
    with pytest.raises(krex.KrexError) as e:
        krex.check_gen_packed(a, torch.float32, 1, 0.0, 0.0)      # no packed stream for fp32
    assert e.value.status == krex.EINVAL
    with pytest.raises(krex.KrexError):
        krex.check_gen_packed(a, torch.float16, 1, 0.0, 0.0, dist="normal", p0=0.0, p1=-1.0)
    with pytest.raises(krex.KrexError):
        krex.check_gen_packed(a, torch.float16, 1, float("inf"), 0.0)


def test_check_gen_packed_at_the_largest_n():
    """n = 2^33 - 1 fp8 elements against the regenerated packed reference:
    zero record for the generated tensor itself, then planted changes on
    both sides of index 2^32 and in the tail give the exact record."""
    n = 2**33 - 1
    a = torch.empty(n, dtype=torch.float8_e4m3fn, device="cuda")
    krex.gen_packed(a, 81, 0, "uniform", -4.0, 4.0)
    r = krex.check_gen_packed(a, torch.float8_e4m3fn, 81, 0.0, 0.0, dist="uniform", p0=-4.0, p1=4.0)
    assert (r.n, r.mismatches, r.nan_count, r.max_abs, r.argmax_abs, r.max_rel) == (n, 0, 0, 0.0, 0, 0.0)
    idx = [7, 2**32 + 3, n - 2]
    v = a.view(torch.uint8)
    before = [float(a[i].float().item()) for i in idx]
    for i in idx:
        v[i] = 0xD8                                    # -16.0
    after = [float(a[i].float().item()) for i in idx]
    r = krex.check_gen_packed(a, torch.float8_e4m3fn, 81, 0.0, 0.0, dist="uniform", p0=-4.0, p1=4.0)
    d = [abs(x - y) for x, y in zip(after, before)]
    assert r.mismatches == 3 and r.nan_count == 0
    assert r.max_abs == max(d) and r.argmax_abs == idx[d.index(max(d))]
    del a
    torch.cuda.empty_cache()
