"""The benchmark configurations at their full sizes, GPU vs oracle:

gemm_tiny     A, B fp32 256 x 256 and the naive GEMM candidate bit for bit,
              and the check against the fp32 reference GEMM (0 mismatches,
              max_abs 0: same k order and fused multiply-adds).
gemm_large    A, B bf16 4096 x 4096 normal(0, 1) bit for bit; the check of a
              bf16 candidate C against an fp32 reference C field for field.
check_stress  x fp16 16384 x 16384 and y = inject(x) bit for bit; the check
              record field for field and against its closed form (max_abs
              exactly 0.5 at the first perturbed index; mismatches = number
              of perturbed elements).
mixed_stream  the 64 derived commands (parameters from GPU words equal the
              oracle's); each command's generated tensor, injected tensor and
              check record against the oracle, on the full tensor up to 2^25
              elements and on windows (offset generation) beyond that."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_30057_amd as krex
from paper_2609_30057_amd import workloads as W
from tests.gpu_helpers import assert_bits_equal, empty, from_storage, same_result, to_storage

pytestmark = pytest.mark.gpu
NAMES = {0: "f32", 1: "bf16", 2: "f16", 3: "f8"}


def test_gemm_tiny():
    cfg = W.GEMM_TINY
    n = cfg["n"]
    offA, offB = W.gemm_tiny_offsets()
    A, B = empty("f32", n * n), empty("f32", n * n)
    krex.gen(A, cfg["seed"], offA, "uniform", -1.0, 1.0)
    krex.gen(B, cfg["seed"], offB, "uniform", -1.0, 1.0)
    Ar = oracle.gen("f32", n * n, cfg["seed"], offA)
    Br = oracle.gen("f32", n * n, cfg["seed"], offB)
    assert_bits_equal(A.cpu().numpy(), Ar, "A")
    assert_bits_equal(B.cpu().numpy(), Br, "B")
    C = torch.empty(n, n, device="cuda")
    krex.fixture_sgemm(A.view(n, n), B.view(n, n), C)
    Cref = oracle.sgemm(Ar.reshape(n, n), Br.reshape(n, n))
    r = krex.check(C.view(-1), from_storage(Cref.ravel(), "f32"), cfg["rtol"], cfg["atol"])
    ref = oracle.check(C.cpu().numpy().ravel(), "f32", Cref.ravel(), "f32", cfg["rtol"], cfg["atol"])
    same_result(r, ref)
    assert r.mismatches == 0 and r.max_abs == 0.0 and r.argmax_abs == 0


def test_gemm_large():
    cfg = W.GEMM_LARGE
    n = cfg["n"]
    offA, offB = W.gemm_large_offsets()
    A, B = empty("bf16", n * n), empty("bf16", n * n)
    krex.gen(A, cfg["seed"], offA, "normal", 0.0, 1.0)
    krex.gen(B, cfg["seed"], offB, "normal", 0.0, 1.0)
    assert_bits_equal(to_storage(A, "bf16"), oracle.gen("bf16", n * n, cfg["seed"], offA, 1, 0.0, 1.0), "A")
    assert_bits_equal(to_storage(B, "bf16"), oracle.gen("bf16", n * n, cfg["seed"], offB, 1, 0.0, 1.0), "B")
    C = torch.matmul(A.view(n, n), B.view(n, n))
    Cref = torch.matmul(A.view(n, n).float(), B.view(n, n).float())
    r = krex.check(C.view(-1), Cref.view(-1), cfg["rtol"], cfg["atol"])
    ref = oracle.check(to_storage(C.view(-1), "bf16"), "bf16", Cref.view(-1).cpu().numpy(), "f32",
                       cfg["rtol"], cfg["atol"])
    same_result(r, ref)


def test_check_stress():
    cfg = W.CHECK_STRESS
    n = cfg["rows"] * cfg["cols"]
    x = empty("f16", n)
    krex.gen(x, cfg["seed"], 0, "uniform", cfg["p0"], cfg["p1"])
    xr = oracle.gen("f16", n, cfg["seed"], 0, 0, cfg["p0"], cfg["p1"])
    assert_bits_equal(to_storage(x, "f16"), xr, "x")
    y = torch.empty_like(x)
    krex.inject(y, x, cfg["mask_seed"], cfg["rate"], cfg["delta"], "exact")
    yr, k = oracle.inject(xr, "f16", cfg["mask_seed"], cfg["rate"], cfg["delta"], oracle.INJ_EXACT)
    assert_bits_equal(to_storage(y, "f16"), yr, "y")
    r = krex.check(y, x, cfg["rtol"], cfg["atol"])
    ref = oracle.check(yr, "f16", xr, "f16", cfg["rtol"], cfg["atol"])
    same_result(r, ref)
    moved = np.nonzero(yr != xr)[0]
    assert r.mismatches == k == moved.size
    assert r.max_abs == 0.5 and r.argmax_abs == moved[0] and r.nan_count == 0
    # 0.1% Bernoulli mask: about 268,435 positions, minus the EXACT-mode drops
    assert 255_000 < k < 262_000


def _mixed_commands_from_gpu():
    w = empty("u32", 1024)
    krex.gen(w, W.MIXED_STREAM["seed"], 0)
    return W.mixed_stream_commands(to_storage(w, "u32"))


def test_mixed_stream_parameters():
    gpu = _mixed_commands_from_gpu()
    ref = W.mixed_stream_commands(oracle.words(1024, W.MIXED_STREAM["seed"], 0))
    assert gpu == ref
    assert all((1 << 20) <= c.size_bytes <= (1 << 30) for c in gpu)
    assert {c.dtype for c in gpu} == {0, 1, 2, 3}


def test_mixed_stream_commands():
    cfg = W.MIXED_STREAM
    for c in _mixed_commands_from_gpu():
        dt = NAMES[c.dtype]
        x = empty(dt, c.n)
        krex.gen(x, c.value_seed, 0, c.dist, c.p0, c.p1)
        y = torch.empty_like(x)
        krex.inject(y, x, c.mask_seed, c.rate, cfg["delta"], "round")
        r = krex.check(y, x, c.rtol, c.atol)
        what = "command %d (%s n=%d)" % (c.index, dt, c.n)
        print(what, flush=True)
        if c.n <= (1 << 25):
            xr = oracle.gen(dt, c.n, c.value_seed, 0, c.dist, c.p0, c.p1)
            assert_bits_equal(to_storage(x, dt), xr, what + " x")
            yr, _ = oracle.inject(xr, dt, c.mask_seed, c.rate, cfg["delta"], oracle.INJ_ROUND)
            assert_bits_equal(to_storage(y, dt), yr, what + " y")
            same_result(r, oracle.check(yr, dt, xr, dt, c.rtol, c.atol))
        else:
            m = 1 << 20
            for start in (0, c.n // 2 + 3, c.n - m):
                xr = oracle.gen(dt, m, c.value_seed, start, c.dist, c.p0, c.p1)
                assert_bits_equal(to_storage(x[start:start + m], dt), xr, what + " x window")
                yr, _ = oracle.inject(xr, dt, c.mask_seed, c.rate, cfg["delta"], oracle.INJ_ROUND, start)
                assert_bits_equal(to_storage(y[start:start + m], dt), yr, what + " y window")
            # the record itself, on the GPU's own tensors copied back: the
            # oracle's check of exactly the bytes the GPU check read
            xs, ys = to_storage(x, dt), to_storage(y, dt)
            same_result(r, oracle.check(ys, dt, xs, dt, c.rtol, c.atol))
            del xs, ys
            assert r.n == c.n and r.nan_count == 0
