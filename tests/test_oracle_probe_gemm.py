"""Pins the oracle's FMA probe by exact rational arithmetic (every fused
multiply-add rounded once to fp32 by hand), and its fp32 reference GEMM by
exact integer inputs and the classical error bound against fp64."""
from fractions import Fraction

import numpy as np


def round_f32(q):
    """Round a rational to the nearest fp32 value, ties to even (normal range)."""
    if q == 0:
        return 0.0
    s = -1 if q < 0 else 1
    q = abs(q)
    e = q.numerator.bit_length() - q.denominator.bit_length()
    while Fraction(2) ** e > q:
        e -= 1
    while Fraction(2) ** (e + 1) <= q:
        e += 1
    e = max(e, -126)
    scale = Fraction(2) ** (23 - e)
    m = q * scale
    fl = m.numerator // m.denominator
    rem = m - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return s * float(Fraction(fl) / scale)


def test_probe_exact_emulation(oracle_mod):
    threads, iters = 24, 40
    got = oracle_mod.probe(iters, threads)
    a = Fraction(1) - Fraction(1, 1024)
    b = Fraction(1, 1024)
    for g in range(threads):
        xs = [Fraction(g * 8 + c, 2**19) for c in range(8)]
        for _ in range(iters):
            xs = [Fraction(round_f32(x * a + b)) for x in xs]
        s = xs[0]
        for c in range(1, 8):
            s = Fraction(round_f32(s + xs[c]))
        assert got[g] == np.float32(float(s)), g


def test_probe_zero_iterations(oracle_mod):
    got = oracle_mod.probe(0, 100)
    g = np.arange(100, dtype=np.float64)
    exp = sum((g * 8 + c) * 2.0**-19 for c in range(8))       # small integers: exact
    assert np.array_equal(got.astype(np.float64), exp)


def test_sgemm_exact_on_integers(oracle_mod):
    rng = np.random.default_rng(0)
    A = rng.integers(-8, 8, (33, 47)).astype(np.float32)
    B = rng.integers(-8, 8, (47, 29)).astype(np.float32)
    C = oracle_mod.sgemm(A, B)
    assert np.array_equal(C, (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float32))


def test_sgemm_error_bound(oracle_mod):
    rng = np.random.default_rng(1)
    M = N = K = 64
    A = rng.uniform(-1, 1, (M, K)).astype(np.float32)
    B = rng.uniform(-1, 1, (K, N)).astype(np.float32)
    C = oracle_mod.sgemm(A, B).astype(np.float64)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    bound = K * 2.0**-24 * (np.abs(A).astype(np.float64) @ np.abs(B).astype(np.float64))
    assert np.all(np.abs(C - ref) <= bound)
