"""Pins the oracle's value transforms: uniform (closed forms and exactness on
power-of-two ranges), its own fp32 ln / sin / cos against fp64 libm over every
input they can receive (2^24 each), Box-Muller composition and the normal
distribution's moments, and the generation layout (element j uses word
offset + j; the normal pair is words (2p, 2p + 1))."""
import numpy as np
import pytest
from scipy import stats


def ulp_err(got, exact):
    """|got - exact| in units of the fp32 ulp at |exact|."""
    ex = np.asarray(exact, dtype=np.float64)
    e = np.floor(np.log2(np.maximum(np.abs(ex), 2.0**-149)))
    ulp = np.exp2(np.maximum(e, -126) - 23)
    return np.abs(np.asarray(got, dtype=np.float64) - ex) / ulp


# ---------------------------------------------------------------- uniform


def test_uniform_closed_forms(oracle_mod):
    assert oracle_mod.uniform(0, -1.0, 1.0) == -1.0
    assert oracle_mod.uniform(0xFF, -1.0, 1.0) == -1.0          # low 8 bits ignored
    assert oracle_mod.uniform(0xFFFFFFFF, -1.0, 1.0) == 1.0 - 2.0**-23
    assert oracle_mod.uniform(0x80000000, -4.0, 4.0) == 0.0
    assert oracle_mod.uniform(0xFFFFFFFF, -4.0, 4.0) == 4.0 - 2.0**-21
    assert oracle_mod.uniform(0x12345678, 3.0, 3.0) == 3.0      # empty range


@pytest.mark.parametrize("lo,hi", [(-1.0, 1.0), (-4.0, 4.0), (0.0, 1.0), (-2.0, 2.0)])
def test_uniform_exact_on_power_of_two_ranges(oracle_mod, lo, hi):
    """For hi - lo = 2^m and |lo| <= hi - lo, lo + (hi - lo) k 2^-24 (a multiple of
    2^(m-24) below 2^m in magnitude)
    is exactly representable, so the two roundings are exact: compare every
    one of the 2^24 values with the fp64 value."""
    k = np.arange(1 << 24, dtype=np.uint32)
    got = oracle_mod.uniform_many(k << 8, lo, hi)
    exact = lo + (hi - lo) * k.astype(np.float64) * 2.0**-24
    assert np.array_equal(got.astype(np.float64), exact)


def test_uniform_general_range_two_roundings(oracle_mod):
    """Non-power-of-two range: the result is fl(lo + fl(fl(hi - lo) u)), which
    numpy float32 arithmetic (IEEE, no contraction) reproduces."""
    w = oracle_mod.words(1 << 20, 99, 0)
    lo, hi = np.float32(0.1), np.float32(0.7)
    got = oracle_mod.uniform_many(w, float(lo), float(hi))
    u = (w >> 8).astype(np.float32) * np.float32(2.0**-24)
    ref = lo + (hi - lo) * u
    assert np.array_equal(got, ref.astype(np.float32))
    assert got.min() >= lo and got.max() < hi


# ---------------------------------------------------------------- own ln, sin, cos


def test_ln_every_input_within_one_ulp(oracle_mod):
    k = np.arange(1, (1 << 24) + 1, dtype=np.float64)
    u1 = (k * 2.0**-24).astype(np.float32)
    got = oracle_mod.ln_many(u1)
    exact = np.log(k * 2.0**-24)
    err = ulp_err(got[:-1], exact[:-1])
    assert err.max() < 1.0, err.max()
    assert got[-1] == 0.0 and not np.signbit(got[-1])       # ln 1 = +0


def test_ln_other_inputs(oracle_mod):
    x = np.array([2.0**-126, 1e-30, 0.001, 0.3, 0.70710677, 0.70710683, 1.4142135, 1.4142137,
                  2.0, 10.0, 1e30, 3.4e38], dtype=np.float32)
    got = oracle_mod.ln_many(x)
    assert ulp_err(got, np.log(x.astype(np.float64))).max() < 1.0


def test_sincos_every_input_within_two_ulp(oracle_mod):
    k = np.arange(1 << 24, dtype=np.uint32)
    s, c = oracle_mod.sincos_many(k)
    ang = 2.0 * np.pi * k.astype(np.float64) / 2**24
    es, ec = np.sin(ang), np.cos(ang)
    es[[0, 1 << 23]] = 0.0
    ec[[1 << 22, 3 << 22]] = 0.0
    assert ulp_err(s, es).max() < 2.0
    assert ulp_err(c, ec).max() < 2.0
    assert np.abs(s).max() <= 1.0 and np.abs(c).max() <= 1.0


def test_sincos_quadrant_points(oracle_mod):
    assert oracle_mod.sincos_2pi_q24(0) == (0.0, 1.0)
    assert oracle_mod.sincos_2pi_q24(1 << 22) == (1.0, 0.0)
    s, c = oracle_mod.sincos_2pi_q24(1 << 23)
    assert s == 0.0 and c == -1.0
    assert oracle_mod.sincos_2pi_q24(3 << 22) == (-1.0, 0.0)
    s, c = oracle_mod.sincos_2pi_q24(1 << 21)                  # 45 degrees
    assert abs(s - np.sqrt(0.5)) < 2**-23 and s == c


def test_rho_every_input(oracle_mod):
    """rho = sqrt(0 - 2 ln u1) within 1.5 ulp of the fp64 value for every u1,
    and +0 (not -0) at u1 = 1."""
    k = np.arange(1, (1 << 24) + 1, dtype=np.uint32)
    w0 = (k - 1) << 8
    pairs = np.stack([w0, np.zeros_like(w0)], axis=1).reshape(-1)
    z = oracle_mod.normal_pairs(pairs)
    rho = z[0::2]                                               # cos(0) = 1 exactly
    exact = np.sqrt(-2.0 * np.log(k.astype(np.float64) * 2.0**-24))
    assert ulp_err(rho[:-1], exact[:-1]).max() < 1.5
    assert rho[-1] == 0.0 and not np.signbit(rho[-1])
    assert rho.max() <= np.sqrt(2 * 24 * np.log(2)) + 1e-6


def test_normal_pair_composition(oracle_mod):
    rng = np.random.default_rng(5)
    w = rng.integers(0, 2**32, 2 * 100000, dtype=np.uint64).astype(np.uint32)
    z = oracle_mod.normal_pairs(w)
    u1 = ((w[0::2] >> 8).astype(np.float64) + 1) * 2.0**-24
    ang = 2 * np.pi * (w[1::2] >> 8).astype(np.float64) * 2.0**-24
    r = np.sqrt(-2 * np.log(u1))
    tol = 4e-7 * np.maximum(r, 1e-30)
    assert np.all(np.abs(z[0::2] - r * np.cos(ang)) <= tol)
    assert np.all(np.abs(z[1::2] - r * np.sin(ang)) <= tol)


def test_normal_distribution(oracle_mod):
    n = 1 << 22
    z = oracle_mod.gen("f32", n, 17, 0, oracle_mod.NORMAL, 0.0, 1.0).astype(np.float64)
    se = 1 / np.sqrt(n)
    assert abs(z.mean()) < 5 * se
    assert abs(z.var() - 1) < 5 * np.sqrt(2) * se
    assert abs(stats.skew(z)) < 5 * np.sqrt(6 / n)
    assert abs(stats.kurtosis(z)) < 5 * np.sqrt(24 / n)
    assert stats.kstest(z[: 1 << 20], "norm").pvalue > 1e-4
    assert abs(np.corrcoef(z[0::2], z[1::2])[0, 1]) < 5 * np.sqrt(2 / n)


def test_normal_mean_std(oracle_mod):
    z = oracle_mod.gen("f32", 1 << 16, 3, 0, oracle_mod.NORMAL, 0.0, 1.0)
    v = oracle_mod.gen("f32", 1 << 16, 3, 0, oracle_mod.NORMAL, 2.5, 0.5)
    ref = np.float32(2.5) + np.float32(0.5) * z
    assert np.array_equal(v, ref)


# ---------------------------------------------------------------- layout


@pytest.mark.parametrize("dt", ["f32", "bf16", "f16", "f8"])
@pytest.mark.parametrize("dist", [0, 1])
def test_offset_shift(oracle_mod, dt, dist):
    """gen(offset = o)[j] == gen(offset = 0)[o + j] for every dtype and
    distribution (the element's word is offset + j)."""
    full = oracle_mod.gen(dt, 5000, 9, 0, dist, -1.0, 1.0)
    for o in (1, 2, 3, 7, 1000):
        part = oracle_mod.gen(dt, 5000 - o, 9, o, dist, -1.0, 1.0)
        assert np.array_equal(part, full[o:])


def test_uniform_gen_is_transform_of_words(oracle_mod):
    w = oracle_mod.words(10000, 42, 77)
    g = oracle_mod.gen("f32", 10000, 42, 77, 0, -1.0, 1.0)
    assert np.array_equal(g, oracle_mod.uniform_many(w, -1.0, 1.0))
    assert np.array_equal(oracle_mod.gen("u32", 10000, 42, 77), w)


def test_normal_gen_uses_word_pairs(oracle_mod):
    w = oracle_mod.words(10000, 42, 0)
    g = oracle_mod.gen("f32", 10000, 42, 0, 1, 0.0, 1.0)
    z = oracle_mod.normal_pairs(w)
    # mean 0 + 1 * z: only the sign of a zero may differ (0 + -0 = +0)
    assert np.array_equal(g, z + np.float32(0.0))


@pytest.mark.parametrize("dt", ["bf16", "f16", "f8"])
def test_narrow_gen_is_rounded_f32_gen(oracle_mod, dt):
    for dist in (0, 1):
        f = oracle_mod.gen("f32", 20000, 8, 3, dist, -4.0, 4.0)
        g = oracle_mod.gen(dt, 20000, 8, 3, dist, -4.0, 4.0)
        assert np.array_equal(g, oracle_mod.from_f32(f, dt))


def test_gen_rejects_bad_arguments(oracle_mod):
    with pytest.raises(ValueError):
        oracle_mod.gen("f32", 10, 0, 2**64 - 5)                # offset + n wraps
    with pytest.raises(ValueError):
        oracle_mod.gen("f32", 10, 0, 0, 7)                     # unknown distribution


def test_bitcast_is_the_word(oracle_mod):
    w = oracle_mod.words(100000, 21, 5)
    g = oracle_mod.gen("f32", 100000, 21, 5, oracle_mod.BITCAST, 0.0, 0.0)
    assert np.array_equal(g.view(np.uint32), w)
    h = oracle_mod.gen("f16", 100000, 21, 5, oracle_mod.BITCAST, 0.0, 0.0)
    assert np.array_equal(h, oracle_mod.from_f32(w.view(np.float32), "f16"))


def test_transform_words_equals_gen(oracle_mod):
    for dist, p0, p1 in ((0, -1.0, 1.0), (1, 0.0, 1.0), (2, 0.0, 0.0)):
        for dt in ("f32", "bf16", "f16", "f8", "u32"):
            w = oracle_mod.words(4096, 77, 0)
            got = oracle_mod.transform_words(dt, w, dist, p0, p1)
            ref = oracle_mod.gen(dt, 4096, 77, 0, dist, p0, p1)
            assert np.array_equal(got.view(np.uint8), ref.view(np.uint8))


def test_gen_parameter_rules(oracle_mod):
    for dist, p0, p1 in ((0, 1.0, -1.0), (0, float("nan"), 1.0), (0, -3e38, 3e38), (1, 0.0, -1.0),
                         (1, float("inf"), 1.0)):
        with pytest.raises(ValueError):
            oracle_mod.gen("f32", 4, 0, 0, dist, p0, p1)
