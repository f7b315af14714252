"""GPU allclose check vs the oracle, field by field at 0 ULP: the hand-derived
golden cases, random inputs with every kind of special value (raw 32-bit
patterns), near-equal inputs with injected mismatches, all 16 dtype pairs,
ragged and tiny sizes, misaligned operands, and repeated calls reusing one
result buffer."""
import numpy as np
import torch
import pytest

import oracle
import paper_2609_30057_amd as krex
from tests.golden.cases import check_cases
from tests.gpu_helpers import empty, from_storage, same_result, to_storage

pytestmark = pytest.mark.gpu

DTS = ["f32", "bf16", "f16", "f8"]
CASES = check_cases()
TOL = {"f32": (1e-4, 1e-5), "bf16": (1.6e-2, 1e-2), "f16": (1e-3, 1e-3), "f8": (0.125, 0.125)}


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_golden(case):
    name, a, dta, b, dtb, rtol, atol, exp = case
    ga, gb = from_storage(a, dta), from_storage(b, dtb)
    r = krex.check(ga, gb, rtol, atol)
    exp = dict(exp, n=a.size)
    same_result(r, exp)


def _near_pair(dta, dtb, n, seed):
    """b a normal(0,1) reference; a = b moved by an injected delta at 2% of
    positions, rounded to dta; a few exact copies and sign flips."""
    bf = oracle.gen("f32", n, seed, 0, 1, 0.0, 1.0)
    af, _ = oracle.inject(bf, "f32", seed + 1, 0.02, 0.01, oracle.INJ_ROUND)
    af = af.copy()
    af[::101] = -af[::101]
    a = oracle.from_f32(af, dta) if dta != "f32" else af
    b = oracle.from_f32(bf, dtb) if dtb != "f32" else bf
    return a, b


@pytest.mark.parametrize("dta", DTS)
@pytest.mark.parametrize("dtb", DTS)
def test_near_inputs_all_dtype_pairs(dta, dtb):
    for n in (1, 5, 17, 1000, 65537, (1 << 20) + 3):
        a, b = _near_pair(dta, dtb, n, 11)
        rtol, atol = TOL[dta]
        ref = oracle.check(a, dta, b, dtb, rtol, atol)
        r = krex.check(from_storage(a, dta), from_storage(b, dtb), rtol, atol)
        same_result(r, ref)


@pytest.mark.parametrize("dta", DTS)
@pytest.mark.parametrize("dtb", DTS)
def test_special_values_all_dtype_pairs(dta, dtb):
    """Raw bit patterns: NaNs, infinities, zeros, subnormals, huge values."""
    n = 300007
    a = oracle.gen(dta, n, 100, 0, 2, 0.0, 0.0)
    b = oracle.gen(dtb, n, 101, 0, 2, 0.0, 0.0)
    b[::7] = a[::7] if dta == dtb else b[::7]
    for rtol, atol in ((0.0, 0.0), (1e-3, 1e-3), (2.0, 1e30)):
        ref = oracle.check(a, dta, b, dtb, rtol, atol)
        r = krex.check(from_storage(a, dta), from_storage(b, dtb), rtol, atol)
        same_result(r, ref)


def test_misaligned_operands_and_tails():
    for dt in DTS:
        n = 70001
        a, b = _near_pair(dt, dt, n + 3, 21)
        ga, gb = from_storage(a, dt), from_storage(b, dt)
        for sa, sb in ((1, 1), (0, 3), (2, 0)):
            m = n - 1
            ref = oracle.check(a[sa:sa + m], dt, b[sb:sb + m], dt, *TOL[dt])
            r = krex.check(ga[sa:sa + m], gb[sb:sb + m], *TOL[dt])
            same_result(r, ref)


def test_empty_and_reused_buffer():
    out = krex.check_result_buffer()
    x = empty("f32", 0)
    r = krex.check(x, x, 0.0, 0.0, out=out)
    assert (r.n, r.mismatches, r.nan_count, r.argmax_abs, r.max_abs, r.max_rel) == (0, 0, 0, 2**64 - 1, 0.0, 0.0)
    # the buffer is overwritten, not accumulated, by later calls
    for seed in (1, 2, 3):
        a, b = _near_pair("f16", "f32", 100000, seed)
        ref = oracle.check(a, "f16", b, "f32", 1e-3, 1e-3)
        same_result(krex.check(from_storage(a, "f16"), from_storage(b, "f32"), 1e-3, 1e-3, out=out), ref)


def test_argmax_tie_goes_to_lowest_index():
    n = 1 << 22
    a = np.zeros(n, dtype=np.float32)
    b = np.zeros(n, dtype=np.float32)
    idx = np.array([3_000_000, 17, 4_000_000, 17 + 2**20])
    a[idx] = 2.0
    r = krex.check(from_storage(a, "f32"), from_storage(b, "f32"), 0.0, 0.0)
    assert r.argmax_abs == 17 and r.max_abs == 2.0 and r.mismatches == 4


def test_identical_large_inputs():
    n = (1 << 26) + 1
    x = empty("f16", n)
    krex.gen(x, 3, 0, "uniform", -4.0, 4.0)
    r = krex.check(x, x, 0.0, 0.0)
    assert (r.mismatches, r.nan_count, r.argmax_abs, r.max_abs, r.max_rel) == (0, 0, 0, 0.0, 0.0)


def _ratio_inputs(kind, n, seed):
    """fp32 (a, b) pairs stressing the max_rel search: ratios rising or
    falling along the tensor, near-ties within one ulp of the ratio, tiny and
    subnormal references, b = 0 and an infinite difference placed late."""
    rng = np.random.default_rng(seed)
    b = rng.uniform(1.0, 2.0, n).astype(np.float32)
    if kind == "rising":
        r = np.linspace(1e-3, 2e-3, n, dtype=np.float64)
    elif kind == "falling":
        r = np.linspace(2e-3, 1e-3, n, dtype=np.float64)
    elif kind == "ties":
        r = np.full(n, 1e-3)
    else:
        r = rng.uniform(0.0, 1e-3, n)
    d = (r * b).astype(np.float32)
    a = (b + d).astype(np.float32)
    if kind == "subnormal":
        b[::3] = (b[::3] * np.float32(2.0 ** -140)).astype(np.float32)   # subnormal references
        a[::3] = (b[::3] * np.float32(1.5)).astype(np.float32)
    if kind == "late_specials":
        b[n - 5] = 0.0
        a[n - 5] = 1e-30
        a[n - 2] = np.float32(3e38)
        b[n - 2] = np.float32(-3e38)                             # difference overflows: ratio +inf
    return a, b


@pytest.mark.parametrize("kind", ["rising", "falling", "ties", "random", "subnormal", "late_specials"])
def test_max_rel_search_matches_oracle(kind):
    """max_rel at 0 ULP where the wave filter of the kernel is exercised hard:
    every chunk raising the maximum, maxima only at the start, exact ratios
    equal to within an ulp across lanes and waves, subnormal references, and
    an infinite ratio in the n mod E tail or just before it."""
    for n in (1003, (1 << 20) + 5):
        a, b = _ratio_inputs(kind, n, 5)
        for dta, dtb in (("f32", "f32"), ("f16", "f32"), ("bf16", "bf16"), ("f8", "f16"), ("f8", "f8")):
            ac = oracle.from_f32(a, dta) if dta != "f32" else a
            bc = oracle.from_f32(b, dtb) if dtb != "f32" else b
            ref = oracle.check(ac, dta, bc, dtb, 1e-3, 1e-5)
            r = krex.check(from_storage(ac, dta), from_storage(bc, dtb), 1e-3, 1e-5)
            same_result(r, ref)


def _f8_pairs(kind, n, seed):
    """fp8 e4m3fn operand pairs for the fp8 x fp8 max_rel filter: every
    ordered pair of finite fp8 codes (b the reference), arranged so the
    filter's bound is tested at its edge -- ratios rising along the index
    (every chunk raises the maximum), falling (the maximum comes first),
    only the pairs of the largest finite ratio below +inf spread over the
    whole array (ties within and across waves), a random arrangement, and
    subnormal references only. Ratios are ordered exactly (fp64 of fp8
    values is exact)."""
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    av = oracle.to_f32(codes, "f8").astype(np.float64)
    A, B = np.meshgrid(codes, codes, indexing="ij")
    Av, Bv = np.meshgrid(av, av, indexing="ij")
    A, B, Av, Bv = A.ravel(), B.ravel(), Av.ravel(), Bv.ravel()
    d = np.abs(Av - Bv)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(d == 0, 0.0, np.where(Bv == 0, np.inf, d / np.abs(Bv)))
    rng = np.random.default_rng(seed)
    if kind == "subnormal":
        keep = (B & 0x78) == 0          # exponent field 0: zero or subnormal references
        A, B, ratio = A[keep], B[keep], ratio[keep]
    if kind in ("rising", "falling", "ties"):
        fin = np.isfinite(ratio)
        A, B, ratio = A[fin], B[fin], ratio[fin]
    if kind == "ties":
        top = ratio.max()
        sel = np.nonzero(ratio == top)[0]
        low = np.nonzero(ratio < top)[0]
        idx = rng.choice(low, n)
        idx[rng.random(n) < 0.01] = rng.choice(sel, 1)[0]
        return A[idx], B[idx]
    if kind == "random":
        idx = rng.integers(0, A.size, n)
        return A[idx], B[idx]
    order = np.argsort(ratio, kind="stable")
    if kind == "falling":
        order = order[::-1]
    if kind == "subnormal":
        order = rng.permutation(A.size)
    pos = (np.arange(n, dtype=np.int64) * order.size) // n
    return A[order[pos]], B[order[pos]]


@pytest.mark.parametrize("kind", ["rising", "falling", "ties", "random", "subnormal"])
def test_max_rel_search_fp8_pairs(kind):
    """fp8 x fp8 is the one pair whose max_rel candidate filter is a single
    product with a rounded-up 1/R (no infinity, no overflow): max_rel and
    every other field at 0 ULP on arrangements of every finite fp8 pair."""
    for n in (1003, (1 << 20) + 5):
        a, b = _f8_pairs(kind, n, 9)
        for rtol, atol in ((1e-3, 1e-5), (0.125, 0.125)):
            ref = oracle.check(a, "f8", b, "f8", rtol, atol)
            r = krex.check(from_storage(a, "f8"), from_storage(b, "f8"), rtol, atol)
            same_result(r, ref)


def test_check_at_the_maximum_size():
    """n = 2^33 - 1 (the largest n the boundary accepts), fp8 operands of
    8 GiB each: three planted differences, two beyond index 2^32; the record
    follows in closed form (mismatch count, the largest difference and its
    index, max_rel)."""
    n = 2**33 - 1
    a = torch.zeros(n, dtype=torch.float8_e4m3fn, device="cuda")
    b = torch.zeros(n, dtype=torch.float8_e4m3fn, device="cuda")
    b8 = b.view(torch.uint8)
    a8 = a.view(torch.uint8)
    # b = 1.0 (0x38) at the planted indices; a = 1.5 (0x3C), 3.0 (0x44), 1.125 (0x39)
    idx = [3, 2**32 + 5, n - 1]
    for i, av in zip(idx, (0x3C, 0x44, 0x39)):
        b8[i] = 0x38
        a8[i] = av
    r = krex.check(a, b, 0.0, 0.0)
    assert (r.n, r.mismatches, r.nan_count) == (n, 3, 0)
    assert r.argmax_abs == 2**32 + 5 and r.max_abs == 2.0 and r.max_rel == 2.0
    del a, b


def test_check_beyond_the_maximum_size_is_rejected():
    x = torch.empty(16, dtype=torch.float32, device="cuda")
    out = krex.check_result_buffer()
    L = krex.lib()
    assert L.krex_check(ctypes_ptr(x), krex.F32, ctypes_ptr(x), krex.F32, 2**33, 0.0, 0.0, ctypes_ptr(out),
                        None) == krex.EINVAL


def ctypes_ptr(t):
    import ctypes
    return ctypes.c_void_p(t.data_ptr())
