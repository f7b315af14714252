"""Pins the oracle's allclose check: hand-derived golden cases, torch.isclose
(an independent implementation of the same predicate) on finite inputs,
and invariants that a dropped term, a swapped operand or a wrong index would
break."""
import math

import numpy as np
import pytest
import torch

from tests.golden.cases import check_cases

CASES = check_cases()


def _same(x, y):
    return (math.isnan(x) and math.isnan(y)) or x == y


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_golden(oracle_mod, case):
    name, a, dta, b, dtb, rtol, atol, exp = case
    r = oracle_mod.check(a, dta, b, dtb, rtol, atol)
    assert r["n"] == a.size
    for k, v in exp.items():
        assert _same(float(r[k]) if isinstance(v, float) else r[k], v), (name, k, r[k], v)


def _finite_pair(rng, n):
    b = rng.standard_normal(n).astype(np.float32)
    a = b + (rng.standard_normal(n) * 1e-3).astype(np.float32)
    far = rng.random(n) < 0.05
    a[far] = b[far] + rng.standard_normal(int(far.sum())).astype(np.float32)
    same = rng.random(n) < 0.1
    a[same] = b[same]
    return a, b


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("rtol,atol", [(1e-3, 1e-3), (1e-4, 1e-5), (0.0, 1e-3), (1e-2, 0.0)])
def test_mismatch_count_matches_torch_isclose(oracle_mod, seed, rtol, atol):
    rng = np.random.default_rng(seed)
    a, b = _finite_pair(rng, 200000)
    r = oracle_mod.check(a, "f32", b, "f32", rtol, atol)
    ta, tb = torch.from_numpy(a), torch.from_numpy(b)
    close = torch.isclose(ta, tb, rtol=float(np.float32(rtol)), atol=float(np.float32(atol)))
    assert r["mismatches"] == int((~close).sum())
    d = np.abs(a - b)
    assert r["max_abs"] == d.max() and r["argmax_abs"] == int(np.argmax(d))


def test_identical_inputs_give_zero(oracle_mod):
    x = oracle_mod.gen("f16", 100000, 1, 0, 0, -4.0, 4.0)
    r = oracle_mod.check(x, "f16", x, "f16", 0.0, 0.0)
    assert (r["mismatches"], r["nan_count"], r["argmax_abs"], r["max_abs"], r["max_rel"]) == (0, 0, 0, 0.0, 0.0)


def test_injected_delta_is_max_abs(oracle_mod):
    """fp32 values on the 2^-21 grid below 4 in magnitude: +0.5 is always exact,
    so with EXACT injection max_abs is exactly 0.5 at the first masked index and
    the mismatch count is the number of masked elements."""
    x = oracle_mod.gen("f32", 300000, 2, 0, 0, -4.0, 4.0)
    y, k = oracle_mod.inject(x, "f32", 3, 0.001, 0.5, oracle_mod.INJ_EXACT)
    masked = np.nonzero(y != x)[0]
    assert k == masked.size > 0
    r = oracle_mod.check(y, "f32", x, "f32", 1e-3, 1e-3)
    assert r["mismatches"] == k
    assert r["max_abs"] == 0.5 and r["argmax_abs"] == masked[0]
    assert r["max_rel"] == np.max(np.float32(0.5) / np.abs(x[masked]))


def test_scaling_by_two(oracle_mod):
    """Scaling a, b and atol by 2 (exact) keeps the verdicts and rel, doubles d."""
    rng = np.random.default_rng(4)
    a, b = _finite_pair(rng, 50000)
    r1 = oracle_mod.check(a, "f32", b, "f32", 1e-3, 1e-4)
    r2 = oracle_mod.check(2 * a, "f32", 2 * b, "f32", 1e-3, 2e-4)
    assert r1["mismatches"] == r2["mismatches"]
    assert r2["max_abs"] == 2 * r1["max_abs"] and r2["argmax_abs"] == r1["argmax_abs"]
    assert r2["max_rel"] == r1["max_rel"]


def test_permutation_keeps_counts_and_maxima(oracle_mod):
    rng = np.random.default_rng(6)
    a, b = _finite_pair(rng, 50000)
    a[::97] = np.nan
    p = rng.permutation(a.size)
    r1 = oracle_mod.check(a, "f32", b, "f32", 1e-3, 1e-3)
    r2 = oracle_mod.check(a[p], "f32", b[p], "f32", 1e-3, 1e-3)
    for k in ("mismatches", "nan_count", "max_abs", "max_rel"):
        assert r1[k] == r2[k]


def test_mixed_dtypes_equal_upcast_f32(oracle_mod):
    """Checking a narrow tensor against fp32 equals checking its exact fp32 upcast."""
    for dt in ("bf16", "f16", "f8"):
        a = oracle_mod.gen(dt, 40000, 8, 0, 1, 0.0, 1.0)
        b = oracle_mod.gen("f32", 40000, 8, 0, 1, 0.0, 1.0)
        r1 = oracle_mod.check(a, dt, b, "f32", 1e-2, 1e-2)
        r2 = oracle_mod.check(oracle_mod.to_f32(a, dt), "f32", b, "f32", 1e-2, 1e-2)
        assert r1 == r2


def test_rejects_bad_tolerances(oracle_mod):
    x = np.zeros(4, dtype=np.float32)
    for rt, at in ((-1.0, 0.0), (0.0, float("nan")), (float("inf"), 0.0)):
        with pytest.raises(ValueError):
            oracle_mod.check(x, "f32", x, "f32", rt, at)


def test_overflowed_difference_matches_torch():
    """torch.isclose never calls an infinite difference close, even when the
    tolerance overflows too."""
    a = np.array([-3.0e38, 3.0e38, 1.0], dtype=np.float32)
    b = np.array([3.0e38, -3.0e38, 1.5], dtype=np.float32)
    for rtol in (2.0, 10.0):
        close = torch.isclose(torch.from_numpy(a), torch.from_numpy(b), rtol=rtol, atol=0.0)
        import oracle
        r = oracle.check(a, "f32", b, "f32", rtol, 0.0)
        assert r["mismatches"] == int((~close).sum()) == 2
