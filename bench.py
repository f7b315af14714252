#!/usr/bin/env python3
"""Benchmark of the benchmarking-command hot path on one MI355X.

A step is one whole large-GEMM benchmarking command (the gemm_large
workload): generate A and B (bf16 4096 x 4096, normal(0, 1), Philox seed 1),
compute the candidate C (bf16) and the fp32 reference C with the library
GEMM as stand-ins for an agent's kernel and reference, check C against the
reference (rtol 1.6e-2, atol 1e-2), then time the candidate in a critical
region: 10 warm-up launches and 200 timed reps, each preceded by a 1 GiB
cache flush (Section 2.1; Section 4.1; Section 4.2 step 5).

Metric: generate + check + flush GB/s = algorithmic bytes of those kernels
(bytes written by generation and flush, bytes read by the check) divided by
their summed device time, measured with HIP events on the stream they run
on. The roofline object is for the dominant kernel (the flush: 200 GiB of
the step's 200.2 GiB). The timed-region inflation half of the metric is
measured by `--fidelity` (Section 6.4, Eq. 1), which prints its own line.

The default line also carries the commands whose bytes are generation and
check rather than flush, at full size: `check_stress` (2 GiB: generation,
injection and check of 268M fp16 elements, separately and with generation
and injection fused, each kernel's fraction of 8 TB/s) and `mixed_stream`
(64 commands, about 73 GB). It then measures the timing half briefly
(`inflation_p95_1ms`: 1 ms probes, 1000 single-shot samples in regions, a
native repeat and 7 gated sibling processes), unless --no-fidelity.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--no-fidelity]
       python bench.py --fidelity [--samples S] [--siblings N] [--warmup-ms W] [--warmup-mode time|clock]
                              [--sessions K] [--durations 0.1,1,10]
                              [--modes control,gated,ungated,frozen,frozen_nopin,torch_gated,torch_ungated]
       python bench.py --kernels          per-kernel throughput on the command shapes
       python bench.py --configs          the other commands: gemm_tiny, check_stress, mixed_stream
       python bench.py --cache-probe      reads warm / after a flush / cold: what the flush evicts
       python bench.py --calib-copy       also time a plain 1 GiB device copy (the
                                          reference kernel for rocprofv3 byte counters)
       python bench.py --valu-rates       issue cost of the vector instructions the kernels
                                          use (cycles per wave64 instruction per SIMD)
"""
import argparse
import json
import os
import sys
import time
import uuid

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
LEAD_PROBE_ITERS = 3200      # about 0.1 ms of k_probe on one MI355X
GIB = 1 << 30
PROFILES = os.path.join(ROOT, "profiles")


def _traffic_for(kernel_key):
    """HBM bytes per launch from the committed rocprofv3 PMC summary, or None
    when it is missing or the kernel source changed since it was taken."""
    path = os.path.join(PROFILES, "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    ent = data.get(kernel_key)
    from paper_2609_30057_amd.profiling import kernel_source_sha
    if not ent or ent.get("source_sha256") != kernel_source_sha(kernel_key.split("/")[0]):
        return None
    return ent.get("hbm_bytes_per_launch")


def host_facts():
    """The host the oracle runs on: logical CPUs, the CPUs this process may
    use, and the CPU model."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"host_cpus": os.cpu_count(), "allowed_cpus": len(os.sched_getaffinity(0)), "cpu_model": model}


class pinned_core:
    """Runs the block on one core of this process's affinity set (the
    highest-numbered one): the calling thread's affinity is set in-process
    and restored afterwards, so the single-threaded oracle stays on one
    core."""

    def __enter__(self):
        self.saved = os.sched_getaffinity(0)
        self.core = max(self.saved)
        os.sched_setaffinity(0, {self.core})
        return self

    def __exit__(self, *exc):
        os.sched_setaffinity(0, self.saved)
        return False


def cpu_baseline(step_bytes, c_bits, cref):
    """The oracle (single-threaded C) on a bounded sample of one step: both
    generated matrices and the full check of the step's own candidate C
    (bf16 bits) against its fp32 reference (host copies), plus 20 of the 200
    1 GiB flushes (host fill of a pre-touched buffer), scaled to one step's
    byte mix. Runs pinned to one core; the check's record must equal the GPU's."""
    with pinned_core() as pc:
        out = _cpu_baseline(step_bytes, c_bits, cref)
    out.update(host_facts())
    out["core"] = pc.core
    return out


def _cpu_baseline(step_bytes, c_bits, cref):
    import numpy as np
    import oracle
    from paper_2609_30057_amd import workloads as W
    cfg = W.GEMM_LARGE
    n2 = cfg["n"] * cfg["n"]
    offA, offB = W.gemm_large_offsets()
    t0 = time.perf_counter()
    A = oracle.gen("bf16", n2, cfg["seed"], offA, 1, 0.0, 1.0)
    B = oracle.gen("bf16", n2, cfg["seed"], offB, 1, 0.0, 1.0)
    t_gen = time.perf_counter() - t0
    t0 = time.perf_counter()
    rec = oracle.check(c_bits, "bf16", cref, "f32", cfg["rtol"], cfg["atol"])
    t_check = time.perf_counter() - t0
    buf = np.zeros(GIB // 4, dtype=np.uint32)
    oracle.flush_fill(buf, 1)                              # first touch, not timed
    sample_flushes = 20
    t0 = time.perf_counter()
    for r in range(sample_flushes):
        oracle.flush_fill(buf, (0x9E3779B9 * (r + 1)) & 0xFFFFFFFF)
    t_flush = (time.perf_counter() - t0) * (cfg["reps"] / sample_flushes)
    total = t_gen + t_check + t_flush
    del buf
    return {
        "value": round(step_bytes / total / 1e9, 3),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": ("one gemm_large step on the host: generation of both 4096x4096 bf16 normal matrices "
                   "(%.2f s), the full 16.8M-element check of the step's bf16 candidate C against its fp32 "
                   "reference (%.2f s), and 20 of the 200 1 GiB flush fills scaled x10 (%.2f s); "
                   "single-threaded C oracle pinned to one core" % (t_gen, t_check, t_flush)),
        "check_record": rec,
    }


def run_gemm_large(steps, warmup, with_cpu):
    import numpy as np
    import torch

    import paper_2609_30057_amd as krex
    from paper_2609_30057_amd import workloads as W

    cfg = W.GEMM_LARGE
    n = cfg["n"]
    n2 = n * n
    offA, offB = W.gemm_large_offsets()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    A = torch.empty(n, n, dtype=torch.bfloat16, device=dev)
    B = torch.empty_like(A)
    C = torch.empty_like(A)
    Cl = torch.empty_like(A)
    Af = torch.empty(n, n, dtype=torch.float32, device=dev)
    Bf = torch.empty_like(Af)
    Cref = torch.empty_like(Af)
    fl = torch.empty(cfg["flush_bytes"] // 4, dtype=torch.int32, device=dev)
    res = krex.check_result_buffer(dev)
    shm = "/krex-bench-%s" % uuid.uuid4().hex[:10]
    krex.attach(0, shm_name=shm)

    gen_bytes = 2 * n2 * 2
    check_bytes = n2 * (2 + 4)
    flush_bytes = cfg["reps"] * cfg["flush_bytes"]
    step_bytes = gen_bytes + check_bytes + flush_bytes

    def candidate():
        torch.matmul(A, B, out=Cl)

    # About 0.1 ms of the probe kernel ahead of the first event: the timed
    # loop ends each step synchronised, so without it the generation events
    # would also time the host's enqueue of the two generation launches.
    lead_sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device=dev)

    def one_step():
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        krex.probe(LEAD_PROBE_ITERS, lead_sink)
        ev[0].record()
        krex.gen(A, cfg["seed"], offA, "normal", 0.0, 1.0)
        ev[1].record()
        krex.gen(B, cfg["seed"], offB, "normal", 0.0, 1.0)
        ev[2].record()
        torch.matmul(A, B, out=C)
        Af.copy_(A)
        Bf.copy_(B)
        torch.matmul(Af, Bf, out=Cref)
        ev[3].record()
        krex.check(C.view(-1), Cref.view(-1), cfg["rtol"], cfg["atol"], out=res, sync=False)
        ev[4].record()
        times, ftimes = krex.time_loop(candidate, cfg["warmup"], cfg["reps"], flush_buf=fl, region=True,
                                       with_flush_times=True)
        verdict = krex.decode_check_result(res)
        return dict(gen_ms=[ev[0].elapsed_time(ev[1]), ev[1].elapsed_time(ev[2])],
                    check_ms=ev[3].elapsed_time(ev[4]), flush_ms=ftimes, loop_ms=times, verdict=verdict)

    for _ in range(warmup):
        one_step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    recs = [one_step() for _ in range(steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    krex.detach()

    gen_ms = np.array([sum(r["gen_ms"]) for r in recs])
    check_ms = np.array([r["check_ms"] for r in recs])
    flush_ms = np.array([f for r in recs for f in r["flush_ms"]])
    kernel_s = (gen_ms.sum() + check_ms.sum() + flush_ms.sum()) / 1e3
    value = steps * step_bytes / kernel_s / 1e9
    flush_gbps = cfg["flush_bytes"] / (flush_ms.mean() / 1e3) / 1e9
    traffic = _traffic_for("k_flush/gemm_large")
    v = recs[-1]["verdict"]
    out = {
        "metric": "gen+check+flush GB/s vs MI355X HBM peak; p95 in-region timing inflation",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(wall / steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": ("gemm_large: A,B bf16 4096x4096 normal(0,1) Philox seed 1 (B at offset 16777216); "
                         "bf16 candidate C vs fp32 reference C checked at rtol 1.6e-2 atol 1e-2; "
                         "10 warm-up + 200 timed reps of the candidate in a critical region, 1 GiB flush "
                         "before each rep"),
            "tensor_dtypes": "A, B, C bf16; reference C f32 (dtype names the arithmetic: fp32 transforms and "
                             "check, u32 Philox)",
            "elements_per_matrix": n2,
            "flush_bytes": cfg["flush_bytes"],
            "reps": cfg["reps"],
            "algorithmic_bytes_per_step": step_bytes,
            "value_basis": ("algorithmic bytes over the summed HIP-event time of the path's own kernels "
                            "(both generations, the check, the 200 flushes); wall_GBps is over the "
                            "step's wall clock, which also runs the candidate GEMM 210 times and the "
                            "fp32 reference GEMM"),
        },
        "roofline": {
            "kernel": "k_flush",
            "bound": "hbm",
            "achieved": round(flush_gbps, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(flush_gbps / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
        },
        "per_kernel": {
            "gen_bf16_normal": {"ms": round(float(gen_ms.mean() / 2), 4),
                                "GBps": round(n2 * 2 / (gen_ms.mean() / 2 / 1e3) / 1e9, 1)},
            "check_bf16_f32": {"ms": round(float(check_ms.mean()), 4),
                               "GBps": round(check_bytes / (check_ms.mean() / 1e3) / 1e9, 1)},
            "flush_1GiB": {"ms": round(float(flush_ms.mean()), 4), "GBps": round(flush_gbps, 1)},
        },
        "wall_GBps": round(steps * step_bytes / wall / 1e9, 2),
        "candidate_median_ms": round(float(np.median(recs[-1]["loop_ms"])), 4),
        "verdict": {"mismatches": v.mismatches, "nan_count": v.nan_count, "max_abs": v.max_abs,
                    "argmax_abs": v.argmax_abs, "max_rel": v.max_rel},
    }
    if with_cpu:
        import numpy as np
        c_bits = C.view(torch.int16).view(-1).cpu().numpy().view(np.uint16)
        cref = Cref.view(-1).cpu().numpy()
        out["cpu_baseline"] = cpu_baseline(step_bytes, c_bits, cref)
        rec = out["cpu_baseline"]["check_record"]
        gpu_rec = {"mismatches": v.mismatches, "nan_count": v.nan_count, "argmax_abs": v.argmax_abs,
                   "max_abs": v.max_abs, "max_rel": v.max_rel}
        out["cpu_baseline"]["check_record_equals_gpu"] = all(rec[k] == x for k, x in gpu_rec.items())
        del out["cpu_baseline"]["check_record"]
    return out


def short_fidelity(samples=1000):
    """The timing-fidelity half of the metric, briefly: P = p95(t / t_native)
    - 1 (Eq. 1) for the 1 ms probe, single-shot inside regions, with 7 sibling
    processes looping the check_stress command off-region through the gate,
    next to a native repeat (P of a second run alone: the spread of
    single-shot timings, the noise floor) and the median-of-10 variant
    (Section 6.6). The full sweep is --fidelity."""
    from paper_2609_30057_amd import fidelity
    try:
        r = fidelity.run(samples=samples, durations_ms=(1.0,), modes=("control", "gated"))
    except Exception as e:   # the throughput line stays valid without it
        return {"value": None, "error": "%s: %s" % (type(e).__name__, e)}
    return {"value": r["P"]["1.0"]["gated"], "unit": "%", "native_repeat": r["P"]["1.0"]["control"],
            "median_of_10": r["P_median_of_10"]["1.0"]["gated"],
            "median_of_10_native_repeat": r["P_median_of_10"]["1.0"]["control"],
            "probe_ms": 1.0, "samples": samples, "siblings": r["siblings"],
            "sibling_GBps": r["sibling_GBps"].get("gated"), "drain_ms_p95": r["drain_ms"]["gated"]["p95"],
            "warmup": r["warmup"], "clock": r["clock"]["1.0"], "target": "<= 1%"}


def run_kernels():
    """Per-kernel throughput on the commands' shapes (median of 20 launches,
    HIP events on the launching stream; includes the launch gaps)."""
    import torch

    import paper_2609_30057_amd as krex

    def t_ms(fn, reps=20, warm=3):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            b.synchronize()
            ts.append(a.elapsed_time(b))
        ts.sort()
        return ts[len(ts) // 2]

    dev = "cuda:0"
    torch.cuda.set_device(0)
    res = {}
    N = 1 << 24

    def rec(name, ms, nbytes):
        res[name] = {"us": round(ms * 1e3, 1), "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                     "frac_hbm": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 3)}

    x16 = torch.empty(N * 16, dtype=torch.float16, device=dev)
    y16 = torch.empty_like(x16)
    a_bf = torch.empty(N, dtype=torch.bfloat16, device=dev)
    b_f32 = torch.empty(N, dtype=torch.float32, device=dev)
    x8 = torch.empty(N * 16, dtype=torch.float8_e4m3fn, device=dev)
    y8 = torch.empty_like(x8)
    xf = torch.empty(N * 4, dtype=torch.float32, device=dev)
    yf = torch.empty_like(xf)
    fl = torch.empty(GIB // 4, dtype=torch.int32, device=dev)
    out = krex.check_result_buffer()
    rec("gen f16 uniform 268M", t_ms(lambda: krex.gen(x16, 2, 0, "uniform", -4.0, 4.0)), x16.numel() * 2)
    rec("gen bf16 normal 16.8M", t_ms(lambda: krex.gen(a_bf, 1, 0, "normal")), N * 2)
    rec("gen f32 normal 16.8M", t_ms(lambda: krex.gen(b_f32, 1, 0, "normal")), N * 4)
    rec("gen f32 uniform 67M", t_ms(lambda: krex.gen(xf, 7, 0)), xf.numel() * 4)
    rec("gen f8 normal 268M", t_ms(lambda: krex.gen(x8, 5, 0, "normal")), x8.numel())
    rec("gen packed f16 uniform 268M", t_ms(lambda: krex.gen_packed(x16, 2, 0, "uniform", -4.0, 4.0)),
        x16.numel() * 2)
    rec("gen packed bf16 normal 16.8M", t_ms(lambda: krex.gen_packed(a_bf, 1, 0, "normal")), N * 2)
    rec("gen packed f8 uniform 268M", t_ms(lambda: krex.gen_packed(x8, 5, 0, "uniform", -4.0, 4.0)), x8.numel())
    rec("gen packed f8 normal 268M", t_ms(lambda: krex.gen_packed(x8, 5, 0, "normal")), x8.numel())
    rec("inject f16 exact 268M", t_ms(lambda: krex.inject(y16, x16, 3, 0.001, 0.5)), x16.numel() * 4)
    rec("gen+inject fused f16 268M", t_ms(lambda: krex.gen_inject(x16, y16, 2, 0, "uniform", -4.0, 4.0, mask_seed=3,
                                                                   rate=0.001, delta=0.5)), x16.numel() * 4)
    krex.inject(y8, x8, 6, 0.01, 0.25, "round")
    krex.inject(yf, xf, 8, 0.01, 0.5)
    rec("check bf16xf32 16.8M", t_ms(lambda: krex.check(a_bf, b_f32, 1.6e-2, 1e-2, out=out, sync=False)), N * 6)
    rec("check f16xf16 268M", t_ms(lambda: krex.check(y16, x16, 1e-3, 1e-3, out=out, sync=False)), x16.numel() * 4)
    rec("check f8xf8 268M", t_ms(lambda: krex.check(y8, x8, 0.125, 0.125, out=out, sync=False)), x8.numel() * 2)
    rec("check f32xf32 67M", t_ms(lambda: krex.check(yf, xf, 1e-4, 1e-5, out=out, sync=False)), xf.numel() * 8)
    # the check against a regenerated reference reads the candidate only
    rec("check_gen f16 vs f16 uniform 268M", t_ms(lambda: krex.check_gen(y16, torch.float16, 2, 1e-3, 1e-3, dist="uniform",
                                                                          p0=-4.0, p1=4.0, out=out, sync=False)),
        x16.numel() * 2)
    rec("check_gen f8 vs f8 normal 268M", t_ms(lambda: krex.check_gen(y8, torch.float8_e4m3fn, 5, 0.125, 0.125,
                                                                       dist="normal", out=out, sync=False)), x8.numel())
    rec("check_gen f32 vs f32 uniform 67M", t_ms(lambda: krex.check_gen(yf, torch.float32, 7, 1e-4, 1e-5, out=out,
                                                                         sync=False)), xf.numel() * 4)
    rec("check_gen bf16 vs f32 normal 16.8M", t_ms(lambda: krex.check_gen(a_bf, torch.float32, 1, 1.6e-2, 1e-2,
                                                                           dist="normal", out=out, sync=False)), N * 2)
    rec("check_gen_packed f16 vs f16 uniform 268M", t_ms(lambda: krex.check_gen_packed(
        y16, torch.float16, 2, 1e-3, 1e-3, dist="uniform", p0=-4.0, p1=4.0, out=out, sync=False)), x16.numel() * 2)
    rec("check_gen_packed f8 vs f8 uniform 268M", t_ms(lambda: krex.check_gen_packed(
        y8, torch.float8_e4m3fn, 5, 0.125, 0.125, dist="uniform", p0=-4.0, p1=4.0, out=out, sync=False)), x8.numel())
    rec("flush 1GiB", t_ms(lambda: krex.flush(fl, 1)), GIB)
    return {"metric": "per-kernel throughput (algorithmic bytes / event time)", "unit": "GB/s",
            "peak_GBps": HBM_PEAK_GBPS, "kernels": res}


def configs_cpu_baseline(cmds):
    """The oracle (single-threaded C) on bounded samples of the other commands,
    with the same byte accounting as the GPU figures."""
    import numpy as np
    import oracle
    from paper_2609_30057_amd import workloads as W
    out = {}

    def t(fn):
        t0 = time.perf_counter()
        r = fn()
        return time.perf_counter() - t0, r

    def flush_s(nbytes, reps, sample):
        buf = np.zeros(nbytes // 4, dtype=np.uint32)
        oracle.flush_fill(buf, 1)                          # first touch, not timed
        dt, _ = t(lambda: [oracle.flush_fill(buf, (0x9E3779B9 * (r + 1)) & 0xFFFFFFFF) for r in range(sample)])
        return dt * reps / sample

    cfg = W.GEMM_TINY
    n2 = cfg["n"] * cfg["n"]
    offA, offB = W.gemm_tiny_offsets()
    tg, (A, B) = t(lambda: (oracle.gen("f32", n2, cfg["seed"], offA), oracle.gen("f32", n2, cfg["seed"], offB)))
    tc, _ = t(lambda: oracle.check(A, "f32", B, "f32", cfg["rtol"], cfg["atol"]))
    tf = flush_s(cfg["flush_bytes"], cfg["reps"], 10)
    nbytes = 2 * n2 * 4 + n2 * 8 + cfg["reps"] * cfg["flush_bytes"]
    out["gemm_tiny"] = {"value": round(nbytes / (tg + tc + tf) / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
                        "sample": "both matrices, one 65,536-element fp32 check, 10 of the 100 512 MiB flush fills "
                                  "scaled x10"}
    cfg = W.CHECK_STRESS
    m = cfg["rows"] * cfg["cols"] // 8
    tg, x = t(lambda: oracle.gen("f16", m, cfg["seed"], 0, 0, cfg["p0"], cfg["p1"]))
    ti, (y, _) = t(lambda: oracle.inject(x, "f16", cfg["mask_seed"], cfg["rate"], cfg["delta"], oracle.INJ_EXACT))
    tc, _ = t(lambda: oracle.check(y, "f16", x, "f16", cfg["rtol"], cfg["atol"]))
    out["check_stress"] = {"value": round(m * 8 / (tg + ti + tc) / 1e9, 3), "unit": "GB/s", "cores": 1,
                           "kind": "oracle", "sample": "the first eighth of the rows (33,554,432 elements): "
                           "generation %.2f s, injection %.2f s, check %.2f s" % (tg, ti, tc)}
    cfg = W.MIXED_STREAM
    sample = [c for c in cmds if c.nbytes <= 64 * (1 << 20)][:8]
    total, secs = 0, 0.0
    for c in sample:
        dtn = W.DTYPE_NAME[c.dtype]
        tg, x = t(lambda: oracle.gen(dtn, c.n, c.value_seed, 0, c.dist, c.p0, c.p1))
        ti, (y, _) = t(lambda: oracle.inject(x, dtn, c.mask_seed, c.rate, cfg["delta"], oracle.INJ_ROUND))
        tc, _ = t(lambda: oracle.check(y, dtn, x, dtn, c.rtol, c.atol))
        secs += tg + ti + tc
        total += c.nbytes * 4
    secs += flush_s(cfg["flush_bytes"], len(sample), 2)
    total += len(sample) * cfg["flush_bytes"]
    out["mixed_stream"] = {"value": round(total / secs / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
                           "sample": "the first %d commands of at most 64 MiB (%s), with one 512 MiB flush each "
                                     "(2 fills timed, scaled)" % (len(sample), ", ".join(str(c.index) for c in sample))}
    return out


def _event():
    import torch
    e = torch.cuda.Event(enable_timing=True)
    e.record()
    return e


def _rate(nbytes, ms):
    gbps = nbytes / (ms / 1e3) / 1e9
    return {"ms": round(ms, 4), "GBps": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 3)}


def measure_check_stress(reps=5, per_kernel=5):
    """The check_stress command at full size (x fp16 16384 x 16384 uniform
    [-4, 4), seed 2; y = EXACT inject(x, mask seed 3, rate 0.001, delta 0.5);
    check(y, x) at rtol = atol = 1e-3), `reps` times each way: generation,
    injection and check as three launches, and generation with injection
    fused (x and y written in one pass) followed by the check. The command's
    time is HIP events around each step's launches, about 0.1 ms of the
    probe kernel ahead of the first event so no event times the host's
    enqueue; medians over the reps. Each kernel's own time is `per_kernel`
    back-to-back launches of it between two events, divided by their count
    (the launch gaps the step figures include are spread over them), median
    over the reps: the figure a kernel trace reports. Algorithmic bytes (the
    method's): generation and injection each write 2n, the check reads 4n,
    8n = 2 GiB per command either way; each kernel's fraction of 8 TB/s counts
    the bytes it moves (injection: x read and y written, 4n)."""
    import numpy as np
    import torch

    import paper_2609_30057_amd as krex
    from paper_2609_30057_amd import workloads as W

    cfg = W.CHECK_STRESS
    m = cfg["rows"] * cfg["cols"]
    dev = torch.device("cuda:0")
    x = torch.empty(m, dtype=torch.float16, device=dev)
    y = torch.empty_like(x)
    res = krex.check_result_buffer(dev)
    lead = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device=dev)

    def gen():
        krex.gen(x, cfg["seed"], 0, "uniform", cfg["p0"], cfg["p1"])

    def inject():
        krex.inject(y, x, cfg["mask_seed"], cfg["rate"], cfg["delta"], "exact")

    def check():
        krex.check(y, x, cfg["rtol"], cfg["atol"], out=res, sync=False)

    def gen_inject():
        krex.gen_inject(x, y, cfg["seed"], 0, "uniform", cfg["p0"], cfg["p1"], mask_seed=cfg["mask_seed"],
                        rate=cfg["rate"], delta=cfg["delta"], mode="exact")

    def per_launch(fn):
        krex.probe(LEAD_PROBE_ITERS, lead)
        a = _event()
        for _ in range(per_kernel):
            fn()
        b = _event()
        b.synchronize()
        return a.elapsed_time(b) / per_kernel

    sep, fus, verdicts, kern = [], [], [], {"gen": [], "inject": [], "check": [], "gen_inject": []}
    for _ in range(reps):
        krex.probe(LEAD_PROBE_ITERS, lead)
        e0 = _event()
        gen()
        e1 = _event()
        inject()
        e2 = _event()
        check()
        e3 = _event()
        v = krex.decode_check_result(res)
        sep.append((e0.elapsed_time(e1), e1.elapsed_time(e2), e2.elapsed_time(e3)))
        krex.probe(LEAD_PROBE_ITERS, lead)
        f0 = _event()
        gen_inject()
        f1 = _event()
        check()
        f2 = _event()
        vf = krex.decode_check_result(res)
        fus.append((f0.elapsed_time(f1), f1.elapsed_time(f2)))
        verdicts.append((v, vf))
        for name, fn in (("gen", gen), ("inject", inject), ("gen_inject", gen_inject), ("check", check)):
            kern[name].append(per_launch(fn))
    tg, ti, tc = (float(np.median([r[k] for r in sep])) for k in range(3))
    tf, tcf = (float(np.median([r[k] for r in fus])) for k in range(2))
    kt = {k: float(np.median(v)) for k, v in kern.items()}
    v, vf = verdicts[-1]
    same = all((a.mismatches, a.nan_count, a.argmax_abs, a.max_abs, a.max_rel)
               == (b.mismatches, b.nan_count, b.argmax_abs, b.max_abs, b.max_rel)
               == (v.mismatches, v.nan_count, v.argmax_abs, v.max_abs, v.max_rel) for a, b in verdicts)
    alg = 8 * m
    out = {
        "workload": ("check_stress: x fp16 16384x16384 uniform[-4,4) seed 2; y = EXACT inject(x, mask seed 3, "
                     "rate 0.001, delta 0.5); check(y, x) rtol 1e-3 atol 1e-3"),
        "algorithmic_bytes": alg,
        "reps": reps,
        "separate": dict(_rate(alg, tg + ti + tc), steps_ms=[round(tg, 4), round(ti, 4), round(tc, 4)]),
        "fused": dict(_rate(alg, tf + tcf), steps_ms=[round(tf, 4), round(tcf, 4)]),
        "kernels": {"gen_f16_uniform": _rate(2 * m, kt["gen"]), "inject_f16_exact": _rate(4 * m, kt["inject"]),
                    "gen_inject_f16": _rate(4 * m, kt["gen_inject"]),
                    "check_f16_f16 (+ final)": _rate(4 * m, kt["check"])},
        "kernels_basis": "%d back-to-back launches between two events, per launch, median of %d" % (per_kernel, reps),
        "verdict": {"mismatches": v.mismatches, "nan_count": v.nan_count, "argmax_abs": v.argmax_abs,
                    "max_abs": v.max_abs, "max_rel": v.max_rel},
        "verdict_same_every_rep_and_path": bool(same),
    }
    del x, y
    return out


def measure_mixed_stream():
    """The mixed_stream command: 64 commands derived from the words of seed 4
    (1 MiB - 1 GiB, the four dtypes, uniform or normal, 0-1% ROUND
    injection with delta 1.0); each runs generation with injection in one
    call, the check with its verdict read back, and a 512 MiB flush. GB/s of
    the algorithmic bytes (4 bytes per byte of tensor: x and y written, both
    read by the check; plus the flush) over the summed event time of the
    command's launches, and over the wall clock (launches and verdict
    readback included)."""
    import numpy as np
    import torch

    import paper_2609_30057_amd as krex
    from paper_2609_30057_amd import workloads as W

    cfg = W.MIXED_STREAM
    dev = torch.device("cuda:0")
    res = krex.check_result_buffer(dev)
    fl512 = torch.empty(cfg["flush_bytes"] // 4, dtype=torch.int32, device=dev)
    w = torch.empty(1024, dtype=torch.int32, device=dev)
    krex.gen(w, cfg["seed"], 0)
    cmds = W.mixed_stream_commands(w.cpu().numpy().view(np.uint32))
    xbuf = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    ybuf = torch.empty_like(xbuf)
    tdt = {0: torch.float32, 1: torch.bfloat16, 2: torch.float16, 3: torch.float8_e4m3fn}
    torch.cuda.synchronize()
    kernel_ms, total, mism = 0.0, 0, 0
    t0 = time.perf_counter()
    for c in cmds:
        xv = xbuf[:c.nbytes].view(tdt[c.dtype])
        yv = ybuf[:c.nbytes].view(tdt[c.dtype])
        e0 = _event()
        krex.gen_inject(xv, yv, c.value_seed, 0, c.dist, c.p0, c.p1, mask_seed=c.mask_seed, rate=c.rate,
                        delta=cfg["delta"], mode="round")
        krex.check(yv, xv, c.rtol, c.atol, out=res, sync=False)
        krex.flush(fl512)
        e1 = _event()
        mism += krex.decode_check_result(res).mismatches
        kernel_ms += e0.elapsed_time(e1)
        total += c.nbytes * 4 + cfg["flush_bytes"]
    wall = time.perf_counter() - t0
    del xbuf, ybuf
    return cmds, {"workload": "mixed_stream: 64 commands from the words of seed 4, 1 MiB-1 GiB, fp32/bf16/fp16/fp8, "
                              "uniform[-1,1) or normal(0,1), ROUND injection 0-1% delta 1.0, 512 MiB flush each",
                  "algorithmic_bytes": total, "GBps": round(total / (kernel_ms / 1e3) / 1e9, 1),
                  "frac_hbm": round(total / (kernel_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 3),
                  "wall_GBps": round(total / wall / 1e9, 1), "commands_per_s": round(len(cmds) / wall, 1),
                  "mismatches_total": int(mism)}


def run_configs(with_cpu=True):
    """The other commands end to end: gemm_tiny (gen + check + 100 reps with a
    512 MiB flush in a region), check_stress (measure_check_stress) and
    mixed_stream (measure_mixed_stream), with the oracle on one core beside
    them."""
    import numpy as np
    import torch

    import paper_2609_30057_amd as krex
    from paper_2609_30057_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    shm = "/krex-cfg-%s" % uuid.uuid4().hex[:10]
    krex.attach(0, shm_name=shm)
    out = {"metric": "per-command gen+check+flush GB/s", "unit": "GB/s", "commands": {}}
    res = krex.check_result_buffer(dev)

    # gemm_tiny
    cfg = W.GEMM_TINY
    n = cfg["n"]
    offA, offB = W.gemm_tiny_offsets()
    A = torch.empty(n, n, device=dev)
    B = torch.empty_like(A)
    C = torch.empty_like(A)
    fl512 = torch.empty(cfg["flush_bytes"] // 4, dtype=torch.int32, device=dev)
    krex.gen(A, cfg["seed"], offA)
    krex.gen(B, cfg["seed"], offB)
    Cref = torch.matmul(A.cpu(), B.cpu()).to(dev)          # the command's fp32 CPU reference
    krex.fixture_sgemm(A, B, C)
    e0 = _event()
    krex.gen(A, cfg["seed"], offA)
    krex.gen(B, cfg["seed"], offB)
    e1 = _event()
    krex.check(C.view(-1), Cref.view(-1), cfg["rtol"], cfg["atol"], out=res, sync=False)
    e2 = _event()
    times, ftimes = krex.time_loop(krex.sgemm_launcher(A, B, C), cfg["warmup"], cfg["reps"], flush_buf=fl512,
                                   region=True, with_flush_times=True)
    v = krex.decode_check_result(res)
    t = (e0.elapsed_time(e1) + e1.elapsed_time(e2) + sum(ftimes)) / 1e3
    nbytes = 2 * n * n * 4 + n * n * 8 + cfg["reps"] * cfg["flush_bytes"]
    out["commands"]["gemm_tiny"] = {"GBps": round(nbytes / t / 1e9, 1), "bytes": nbytes,
                                    "candidate_median_ms": round(float(np.median(times)), 4),
                                    "mismatches": v.mismatches, "max_abs": v.max_abs}
    del A, B, C, Cref, fl512
    out["commands"]["check_stress"] = measure_check_stress()
    cmds, out["commands"]["mixed_stream"] = measure_mixed_stream()
    krex.detach()
    if with_cpu:
        with pinned_core() as pc:
            for k, v in configs_cpu_baseline(cmds).items():
                v.update(host_facts())
                v["core"] = pc.core
                out["commands"][k]["cpu_baseline"] = v
    return out


def run_hbm_commands():
    """The two commands whose bytes are generation and check rather than
    flush, at full size, attached and gated like any command:
    check_stress (2 GiB of generation, injection and check) and
    mixed_stream (64 commands, about 73 GB)."""
    import torch

    import paper_2609_30057_amd as krex
    torch.cuda.set_device(0)
    krex.attach(0, shm_name="/krex-hbm-%s" % uuid.uuid4().hex[:10])
    try:
        cs = measure_check_stress()
        _, ms = measure_mixed_stream()
    finally:
        krex.detach()
    return {"check_stress": cs, "mixed_stream": ms}


def run_cache_probe(reps=11):
    """What the cache flush must evict, measured: reads (torch's sum, ordinary
    loads that allocate in the caches) of a 64 MiB buffer x timed with HIP
    events in three states:
      warm     x was read by the launch just before (it fits in the 256 MB
               Infinity Cache);
      flushed  a 1 GiB flush (k_flush) ran between the two reads;
      cold     64 MiB slices of a 2 GiB buffer, written in order and then
               read in order, so at least 1.9 GiB of other traffic separates
               each slice's last touch from its read (no cache can hold it);
    and, for the L2, a 2 MiB buffer read twice in a row (it fits in every
    XCD's 4 MB L2): under `rocprofv3 --pmc TCC_HIT_sum TCC_MISS_sum` the
    second read's hits show whether L2 contents survive a kernel boundary.
    Each measured read is preceded by a one-iteration probe launch that marks
    it in a kernel trace."""
    import numpy as np
    import torch

    import paper_2609_30057_amd as krex
    torch.cuda.set_device(0)
    dev = "cuda:0"
    x = torch.ones(16 << 20, dtype=torch.float32, device=dev)
    fl = torch.empty(GIB // 4, dtype=torch.int32, device=dev)
    W = torch.empty(32, 16 << 20, dtype=torch.float32, device=dev)
    small = torch.ones(1 << 19, dtype=torch.float32, device=dev)
    sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device=dev)

    def timed(t):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        krex.probe(1, sink)
        a.record()
        t.sum()
        b.record()
        b.synchronize()
        return a.elapsed_time(b)

    for _ in range(5):
        timed(x)
    warm, flushed, cold = [], [], []
    for _ in range(reps):
        x.sum()
        warm.append(timed(x))
        krex.flush(fl, 7)
        flushed.append(timed(x))
    W.fill_(1.0)
    for k in range(min(reps, 32)):
        cold.append(timed(W[k]))
    small.sum()
    l2 = [timed(small) for _ in range(3)]
    med = {k: float(np.median(v)) for k, v in (("warm", warm), ("flushed", flushed), ("cold", cold))}
    mib = 64 * (1 << 20)
    return {"metric": "64 MiB read time (ms) by cache state; GB/s", "reps": reps,
            "ms": {k: round(v, 4) for k, v in med.items()},
            "GBps": {k: round(mib / (v / 1e3) / 1e9, 1) for k, v in med.items()},
            "flushed_over_cold": round(med["flushed"] / med["cold"], 3),
            "warm_over_cold": round(med["warm"] / med["cold"], 3),
            "l2_small_read_ms": [round(v, 4) for v in l2]}


def run_copy_calibration():
    """A plain device-to-device copy of 1 GiB, three times: the kernel whose
    rocprofv3 FETCH_SIZE / WRITE_SIZE readings calibrate the byte counters."""
    import torch
    src = torch.ones(GIB // 4, dtype=torch.int32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-fidelity", action="store_true",
                    help="skip the short 1 ms in-region inflation measurement of the default run")
    ap.add_argument("--fidelity", action="store_true")
    ap.add_argument("--samples", type=int, default=None)
    ap.add_argument("--siblings", type=int, default=None, help="fidelity sibling processes (default 7)")
    ap.add_argument("--warmup-ms", type=float, default=None,
                    help="fidelity: in-region warm-up time per sample (default 3 ms; 0: one warm-up launch)")
    ap.add_argument("--warmup-mode", default=None, choices=("time", "clock"),
                    help="fidelity: warm up until the probe's slowest-wave clock reaches its calibration median "
                         "(clock, the default), or for a fixed time (time)")
    ap.add_argument("--clock-cap-ms", type=float, default=None,
                    help="fidelity: longest clock warm-up per sample (default 20 ms)")
    ap.add_argument("--lead", type=int, default=None,
                    help="fidelity, clock warm-up: probe launches enqueued without a wait right before each "
                         "sample's flush and timed launch (default from the workload)")
    ap.add_argument("--sessions", type=int, default=1, help="fidelity: repeats of the compared modes")
    ap.add_argument("--dump", default=None, help="fidelity: .npz path for every sample's time and clocks")
    ap.add_argument("--durations", default=None, help="fidelity: probe durations in ms, comma-separated")
    ap.add_argument("--modes", default=None,
                    help="fidelity modes, comma-separated from control,gated,ungated,frozen")
    ap.add_argument("--kernels", action="store_true")
    ap.add_argument("--calib-copy", action="store_true")
    ap.add_argument("--only-gemm-large", action="store_true",
                    help="the gemm_large command alone, without the check_stress and mixed_stream blocks "
                         "(for profiling its kernels)")
    ap.add_argument("--configs", action="store_true")
    ap.add_argument("--cache-probe", action="store_true",
                    help="64 MiB reads warm / after a 1 GiB flush / cold, and an L2 re-read (rocprofv3 --pmc)")
    ap.add_argument("--valu-rates", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (use --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if args.fidelity:
        from paper_2609_30057_amd import fidelity
        modes = args.modes.split(",") if args.modes else None
        print(json.dumps(fidelity.run(samples=args.samples, modes=modes, siblings=args.siblings,
                                      warmup_ms=args.warmup_ms, warmup=args.warmup_mode, sessions=args.sessions,
                                      clock_cap_ms=args.clock_cap_ms, lead=args.lead,
                                      durations_ms=tuple(float(x) for x in args.durations.split(","))
                                      if args.durations else None, dump=args.dump)), flush=True)
        return
    if args.kernels:
        out = run_kernels()
        if args.calib_copy:
            run_copy_calibration()
        print(json.dumps(out), flush=True)
        return
    if args.cache_probe:
        print(json.dumps(run_cache_probe()), flush=True)
        return
    if args.configs:
        print(json.dumps(run_configs(not args.no_cpu_baseline)), flush=True)
        return
    if args.valu_rates:
        import subprocess
        exe = os.path.join(ROOT, "paper_2609_30057_amd", "valu_rates")
        if not os.path.exists(exe):
            raise SystemExit("valu_rates is not built; run __graft_entry__.build()")
        sys.exit(subprocess.run([exe]).returncode)
    out = run_gemm_large(args.steps, args.warmup, not args.no_cpu_baseline)
    if not args.only_gemm_large:
        out.update(run_hbm_commands())
    if args.calib_copy:
        run_copy_calibration()
    if not args.no_fidelity:
        out["inflation_p95_1ms"] = short_fidelity()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
