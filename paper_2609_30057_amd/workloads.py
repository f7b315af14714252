"""The synthetic benchmarking commands this hot path is measured on.

The paper replays recorded agent commands (KernelBench, Atrex-Bench,
FlashInfer-Trace; Section 6.1) that are not available here. These seeded,
synthetic commands stand in for them, with the shapes of a GEMM candidate's
benchmarking command (Section 2.1, Fig. 1a: generate, check, then a timed
loop with cache flushes) and of a check-heavy and a mixed stream of commands.

  gemm_tiny      A, B fp32 256 x 256 uniform[-1, 1), seed 0 (B at offset
                 65536); naive fp32 GEMM candidate vs an fp32 reference;
                 rtol 1e-4, atol 1e-5; 100 timed reps, 512 MiB flush.
  gemm_large     A, B bf16 4096 x 4096 normal(0, 1), seed 1 (B at offset
                 4096^2); bf16 candidate C checked against an fp32 reference
                 C, rtol 1.6e-2, atol 1e-2; 200 timed reps, 1 GiB flush.
  check_stress   x fp16 16384 x 16384 uniform[-4, 4), seed 2; y = x with a
                 0.1% Bernoulli mask (mask seed 3) moved by exactly 0.5;
                 check(y, x) at rtol = atol = 1e-3.
  shared         one prober timing 0.1 / 1 / 10 ms FMA probes inside regions
                 while 7 processes run check_stress generate + check work.
  mixed_stream   64 commands derived from the words of seed 4
                 (mixed_stream_commands).
"""
from dataclasses import dataclass

MIB = 1 << 20
GIB = 1 << 30

F32, BF16, F16, F8E4M3 = 0, 1, 2, 3
ITEMSIZE = {F32: 4, BF16: 2, F16: 2, F8E4M3: 1}
DTYPE_NAME = {F32: "f32", BF16: "bf16", F16: "f16", F8E4M3: "f8"}

# Per-dtype tolerances of the mixed stream: fp32 and bf16 from the two GEMM
# commands, fp16 from the check-stress command, fp8 at e4m3's relative
# spacing 2^-3.
TOLERANCES = {F32: (1e-4, 1e-5), BF16: (1.6e-2, 1e-2), F16: (1e-3, 1e-3), F8E4M3: (0.125, 0.125)}

GEMM_TINY = dict(name="gemm_tiny", n=256, dtype=F32, dist=0, p0=-1.0, p1=1.0, seed=0, rtol=1e-4, atol=1e-5,
                 reps=100, warmup=10, flush_bytes=512 * MIB)
GEMM_LARGE = dict(name="gemm_large", n=4096, dtype=BF16, dist=1, p0=0.0, p1=1.0, seed=1, rtol=1.6e-2, atol=1e-2,
                  reps=200, warmup=10, flush_bytes=GIB)
CHECK_STRESS = dict(name="check_stress", rows=16384, cols=16384, dtype=F16, dist=0, p0=-4.0, p1=4.0, seed=2,
                    mask_seed=3, rate=0.001, delta=0.5, mode=1, rtol=1e-3, atol=1e-3)
# warmup: in-region warm-up of the probe before the flush and the timed
# launch (do_bench warms up before timing, Section 8). "clock": launches one
# at a time until the slowest wave's shader clock reaches the median the
# probe ran at in calibration (at most clock_cap_ms). On one MI355X a probe
# launch lasts its waves' fixed cycle count over the slowest XCD's clock plus
# a constant 3.8 us, and a region entered right after the siblings' memory
# load starts 1-1.4% below the clock of an idle device; the clock warm-up
# removes that difference, where a fixed 3 ms of warm-up ("time", warmup_ms)
# leaves it.
SHARED = dict(name="shared", probe_ms=(0.1, 1.0, 10.0), siblings=7, samples=1000, flush_bytes=512 * MIB,
              gap_ms=5.0, warmup="clock", warmup_ms=3.0, clock_cap_ms=20.0, chunk_bytes=64 * MIB)
MIXED_STREAM = dict(name="mixed_stream", commands=64, seed=4, delta=1.0, mode=0, flush_bytes=512 * MIB)


@dataclass
class Command:
    index: int
    size_bytes: int
    dtype: int
    n: int
    dist: int          # 0 uniform[-1, 1), 1 normal(0, 1)
    rate: float
    value_seed: int
    mask_seed: int
    rtol: float
    atol: float

    @property
    def p0(self):
        return -1.0 if self.dist == 0 else 0.0

    @property
    def p1(self):
        return 1.0

    @property
    def nbytes(self):
        return self.n * ITEMSIZE[self.dtype]


def _u(w):
    return (int(w) >> 8) * 2.0**-24


def mixed_stream_commands(words):
    """The 64 commands of the mixed stream from the words W_4[0 .. 1024):
    command k reads words 16k .. 16k + 7: size 2^(20 + 10 U0) bytes
    (log-uniform 1 MiB - 1 GiB), dtype W1 >> 30, distribution W2 >> 31,
    mismatch rate 0.01 U3, value seed W4 | W5 << 32, mask seed W6 | W7 << 32,
    with U(W) = (W >> 8) 2^-24."""
    cmds = []
    for k in range(MIXED_STREAM["commands"]):
        w = [int(x) for x in words[16 * k:16 * k + 8]]
        size = int(2.0 ** (20.0 + 10.0 * _u(w[0])))
        dt = w[1] >> 30
        n = max(1, size // ITEMSIZE[dt])
        dist = w[2] >> 31
        rate = 0.01 * _u(w[3])
        rtol, atol = TOLERANCES[dt]
        cmds.append(Command(k, size, dt, n, dist, rate, w[4] | (w[5] << 32), w[6] | (w[7] << 32), rtol, atol))
    return cmds


def gemm_large_offsets():
    n = GEMM_LARGE["n"] * GEMM_LARGE["n"]
    return 0, n


def gemm_tiny_offsets():
    n = GEMM_TINY["n"] * GEMM_TINY["n"]
    return 0, n
