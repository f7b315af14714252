"""Pins the oracle's mismatch injection: the Bernoulli threshold's closed
form, the mask as a function of the (independently pinned) Philox words,
ROUND mode against numpy's IEEE float32 add and RNE float16 cast, and EXACT
mode against a brute-force decision made in exact float64 arithmetic over
the fp16 grid."""
import numpy as np
import pytest


def test_threshold_closed_forms(oracle_mod):
    assert oracle_mod.inject_threshold(0.0) == 0
    assert oracle_mod.inject_threshold(1.0) == 2**32
    assert oracle_mod.inject_threshold(0.5) == 2**31
    assert oracle_mod.inject_threshold(0.001) == 4294967        # floor(4294967.296)
    assert oracle_mod.inject_threshold(0.01) == 42949672        # floor(42949672.96)
    assert oracle_mod.inject_threshold(2.0**-32) == 1
    assert oracle_mod.inject_threshold(1e-10) == 0


def test_rate_zero_and_one(oracle_mod):
    x = oracle_mod.gen("f16", 10000, 1, 0, 0, -4.0, 4.0)
    y, k = oracle_mod.inject(x, "f16", 3, 0.0, 0.5, oracle_mod.INJ_ROUND)
    assert k == 0 and np.array_equal(y, x)
    y, k = oracle_mod.inject(x, "f16", 3, 1.0, 0.5, oracle_mod.INJ_ROUND)
    assert k == x.size


@pytest.mark.parametrize("moff", [0, 3, 12345])
def test_mask_is_word_threshold(oracle_mod, moff):
    n = 200000
    x = oracle_mod.gen("f32", n, 2, 0, 0, -4.0, 4.0)
    y, k = oracle_mod.inject(x, "f32", 3, 0.01, 0.5, oracle_mod.INJ_EXACT, mask_offset=moff)
    w = oracle_mod.words(n, 3, moff)
    mask = w.astype(np.uint64) < oracle_mod.inject_threshold(0.01)
    assert np.array_equal(y != x, mask)
    assert k == mask.sum()
    assert np.all(y[mask] - x[mask] == np.float32(0.5))       # fp32: +0.5 always exact here


def test_round_mode_matches_numpy(oracle_mod):
    n = 100000
    for dt, npdt in (("f16", np.float16), ("f32", np.float32)):
        x = oracle_mod.gen(dt, n, 4, 0, 1, 0.0, 1.0)
        y, k = oracle_mod.inject(x, dt, 5, 0.02, 1.0, oracle_mod.INJ_ROUND)
        xf = x.view(np.float16).astype(np.float32) if dt == "f16" else x
        mask = oracle_mod.words(n, 5, 0).astype(np.uint64) < oracle_mod.inject_threshold(0.02)
        ref = xf.copy()
        ref[mask] = xf[mask] + np.float32(1.0)
        ref = ref.astype(npdt)
        got = y.view(np.float16) if dt == "f16" else y
        assert np.array_equal(got.view(np.uint16 if dt == "f16" else np.uint32),
                              ref.view(np.uint16 if dt == "f16" else np.uint32))
        assert k == mask.sum()


def test_exact_mode_fp16_brute_force(oracle_mod):
    """Every masked element becomes x + 0.5 if that is an fp16 value, else
    x - 0.5 if that is, else stays x; decided here in exact float64
    arithmetic over the fp16 grid."""
    n = 1 << 21
    x = oracle_mod.gen("f16", n, 2, 0, 0, -4.0, 4.0)
    y, k = oracle_mod.inject(x, "f16", 3, 0.01, 0.5, oracle_mod.INJ_EXACT)
    mask = oracle_mod.words(n, 3, 0).astype(np.uint64) < oracle_mod.inject_threshold(0.01)
    xv = x.view(np.float16).astype(np.float64)
    plus, minus = xv + 0.5, xv - 0.5
    rep_plus = plus.astype(np.float16).astype(np.float64) == plus
    rep_minus = minus.astype(np.float16).astype(np.float64) == minus
    exp = np.where(rep_plus, plus, np.where(rep_minus, minus, xv))
    exp = np.where(mask, exp, xv).astype(np.float16)
    assert np.array_equal(y, exp.view(np.uint16))
    dropped = mask & ~rep_plus & ~rep_minus
    assert k == int(mask.sum() - dropped.sum())
    assert dropped.sum() > 0 and np.all(np.abs(xv[dropped]) < 0.25)


def test_exact_mode_fp8_and_bf16_only_exact_moves(oracle_mod):
    for dt in ("f8", "bf16"):
        x = oracle_mod.gen(dt, 100000, 6, 0, 1, 0.0, 1.0)
        y, k = oracle_mod.inject(x, dt, 7, 0.05, 0.25, oracle_mod.INJ_EXACT)
        xf, yf = oracle_mod.to_f32(x, dt).astype(np.float64), oracle_mod.to_f32(y, dt).astype(np.float64)
        moved = xf != yf
        assert moved.sum() == k
        assert np.all(np.abs(yf[moved] - xf[moved]) == 0.25)


def test_in_place_alias(oracle_mod):
    """y may alias x; the C oracle supports it and the wrapper writes a copy."""
    x = oracle_mod.gen("f16", 5000, 1, 0, 0, -4.0, 4.0)
    y1, _ = oracle_mod.inject(x, "f16", 3, 0.1, 0.5, oracle_mod.INJ_EXACT)
    import ctypes
    z = x.copy()
    oracle_mod.lib().ko_inject(ctypes.c_void_p(z.ctypes.data), ctypes.c_void_p(z.ctypes.data), 2, z.size,
                               3, 0, 0.1, 0.5, 1)
    assert np.array_equal(z, y1)


def test_rejects_bad_arguments(oracle_mod):
    x = np.zeros(8, dtype=np.float32)
    for rate in (-0.1, 1.5, float("nan")):
        with pytest.raises(ValueError):
            oracle_mod.inject(x, "f32", 1, rate, 0.5)
