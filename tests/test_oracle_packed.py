"""Pins the oracle's packed stream (the narrow-dtype generator that spends
16 or 8 bits of the Philox word stream per element) to things outside its
own arithmetic: the bitcast form is the little-endian byte view of the word
stream; every uniform value equals lo + (hi - lo) f 2^-w rounded twice to
fp32 (computed here with exact rationals and an explicit round-to-nearest-
even) and narrowed by torch; every normal value sits at the radius and angle
that fp64 libm gives for its field pair (cosine on even fields, sine on
odd); the normal samples have N(0, 1) moments; and generating at an offset
is a slice of generating from 0."""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

F16, BF16, F8 = "f16", "bf16", "f8"
TORCH = {F16: torch.float16, BF16: torch.bfloat16, F8: torch.float8_e4m3fn}


def fields(dt, dist, n, seed, offset):
    """Field values of the packed stream, read off the bitcast form's width
    as a byte view of the plain word stream (independent of the oracle's
    field extraction)."""
    w = oracle.packed_width(dt, dist)
    k = 32 // w
    first = offset // k
    words = oracle.words((offset + n + k - 1) // k - first + 1, seed, first)
    view = words.view(np.uint16 if w == 16 else np.uint8)
    s = offset - first * k
    return view[s:s + n].astype(np.int64), w


def round_f32(x):
    """Exact rational -> nearest fp32, ties to even."""
    c = np.float32(float(x))
    best = None
    for cand in (np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))):
        d = abs(Fraction(float(cand)) - x)
        key = (d, int(np.float32(cand).view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, cand)
    return np.float32(best[1])


def narrow(v32, dt):
    t = torch.from_numpy(np.asarray(v32, dtype=np.float32)).to(TORCH[dt])
    return t.view(torch.uint8 if dt == F8 else torch.int16).numpy().view(np.uint8 if dt == F8 else np.uint16)


@pytest.mark.parametrize("dt", [F16, BF16, F8])
@pytest.mark.parametrize("offset", [0, 1, 3, 7, 4097])
def test_bitcast_is_the_byte_view_of_the_word_stream(dt, offset):
    for n in (1, 5, 64, 1001):
        got = oracle.gen_packed(dt, n, 17, offset, oracle.BITCAST)
        f, w = fields(dt, oracle.BITCAST, n, 17, offset)
        assert w == (8 if dt == F8 else 16)
        assert np.array_equal(got.astype(np.int64), f)


@pytest.mark.parametrize("dt", [F16, BF16, F8])
@pytest.mark.parametrize("lo,hi", [(-4.0, 4.0), (-1.0, 1.0), (0.0, 1.0), (-3.0, 7.5), (0.1, 0.3)])
def test_uniform_values_match_exact_rounding(dt, lo, hi):
    """Each field value f maps to RN(lo + RN((hi - lo) f 2^-w)); a long stream
    covers every field value."""
    n = 1 << 20 if dt != F8 else 1 << 14
    got = oracle.gen_packed(dt, n, 5, 3, oracle.UNIFORM, lo, hi)
    f, w = fields(dt, oracle.UNIFORM, n, 5, 3)
    assert len(np.unique(f)) == (1 << w)            # every field value occurs
    lo32, hi32 = np.float32(lo), np.float32(hi)
    r = round_f32(Fraction(float(hi32)) - Fraction(float(lo32)))
    table = np.empty(1 << w, dtype=np.float32)
    for v in range(1 << w):
        t = round_f32(Fraction(float(r)) * Fraction(v, 1 << w))
        table[v] = round_f32(Fraction(float(lo32)) + Fraction(float(t)))
    exp = narrow(table[f], dt)
    assert np.array_equal(got, exp)


@pytest.mark.parametrize("dt", [F16, BF16, F8])
def test_normal_radius_and_angle_follow_the_field_pair(dt):
    """Element q takes rho cos(2 pi a) (q even) or rho sin(2 pi a) (q odd) with
    rho = sqrt(-2 ln u1), u1 = (256 f_{2p} + 1) 2^-24, a = f_{2p+1} 2^-16,
    p = q >> 1: checked in fp64 to within the narrowed format's precision."""
    n, off = 200000, 6
    got = oracle.gen_packed(dt, n, 9, off, oracle.NORMAL, 0.0, 1.0)
    v = torch.from_numpy(got.view(np.uint8 if dt == F8 else np.int16)).view(TORCH[dt]).float().numpy()
    f, w = fields(dt, oracle.NORMAL, n + 2, 9, off - (off & 1))   # whole pairs from the even field below off
    assert w == 16
    pair_lo = f[0::2][: (n + 2) // 2]
    pair_hi = f[1::2][: (n + 2) // 2]
    q = off + np.arange(n)
    p = (q >> 1) - (off >> 1)
    u1 = (256.0 * pair_lo[p] + 1.0) * 2.0**-24
    a = pair_hi[p] * 2.0**-16
    rho = np.sqrt(-2.0 * np.log(u1))
    exp = np.where(q & 1, rho * np.sin(2 * np.pi * a), rho * np.cos(2 * np.pi * a))
    rel = {F16: 2.0**-10, BF16: 2.0**-7, F8: 2.0**-3}[dt]
    tiny = {F16: 2.0**-23, BF16: 2.0**-120, F8: 2.0**-9}[dt]
    assert np.all(np.abs(v - exp) <= rel * np.abs(exp) + tiny + 1e-6 * rho)


def test_normal_moments():
    n = 1 << 20
    v = torch.from_numpy(oracle.gen_packed(F16, n, 21, 0, oracle.NORMAL, 0.0, 1.0).view(np.int16))
    z = v.view(torch.float16).double().numpy()
    assert abs(z.mean()) < 5 * n**-0.5
    assert abs(z.var() - 1.0) < 5 * (2.0 / n) ** 0.5
    assert np.abs(z).max() < 5.8                    # u1 >= 2^-24 bounds the radius by sqrt(48 ln 2)
    mu, sigma = 2.5, 0.5
    v2 = torch.from_numpy(oracle.gen_packed(F16, n, 21, 0, oracle.NORMAL, mu, sigma).view(np.int16))
    z2 = v2.view(torch.float16).double().numpy()
    assert abs(z2.mean() - mu) < 5 * sigma * n**-0.5


@pytest.mark.parametrize("dt,dist", [(F16, oracle.UNIFORM), (BF16, oracle.NORMAL), (F8, oracle.UNIFORM),
                                     (F8, oracle.NORMAL), (F8, oracle.BITCAST)])
def test_offset_is_a_slice(dt, dist):
    full = oracle.gen_packed(dt, 3000, 4, 0, dist, 0.0, 1.0)
    for off in (1, 2, 5, 8, 17, 1023):
        assert np.array_equal(oracle.gen_packed(dt, 3000 - off, 4, off, dist, 0.0, 1.0), full[off:])


def test_rejections():
    for dt in ("f32", "u32"):
        with pytest.raises(ValueError):
            oracle.gen_packed(dt, 4, 1, 0, oracle.UNIFORM, 0.0, 1.0)
    with pytest.raises(ValueError):
        oracle.gen_packed(F16, 4, 1, 0, oracle.UNIFORM, 1.0, 0.0)
    with pytest.raises(ValueError):
        oracle.gen_packed(F16, 4, 1, 0, oracle.NORMAL, 0.0, -1.0)
    with pytest.raises(ValueError):
        oracle.gen_packed(F16, 2, 1, 2**64 - 1, oracle.UNIFORM, 0.0, 1.0)
