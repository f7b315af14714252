"""Shared-GPU timing fidelity: p95 inflation of probe kernels timed inside
critical regions while sibling processes generate and check on the same GPU.

Paper: Section 6.4 (Eq. 1, P = p95(t_measured / t_native) - 1, with a second
native run as the control for run-to-run noise, and fidelity by kernel
duration, 0.1 / 1 / 10 ms); Section 6.5 (ungated sharing as the
unprotected baseline); Section 6.6 (single-shot and median-of-ten timing).

Procedure, on one GPU:
  0. settle: probe launches back to back for about 2 s, so the device's
     clock and thermal state after earlier work (a benchmark just before)
     does not drift between the native run and the later ones;
  1. calibrate the probe's iteration count to each target duration, alone;
  2. native: `samples` single-shot timings per duration, alone (each sample:
     region entry, warm-up launches for about 3 ms (or exactly one with
     warmup_ms = 0), a 512 MiB flush, one timed launch, exit; then a 5 ms
     off-region gap);
  3. control: the same again (native repeat);
  4. gated: the same while `siblings` processes loop generate -> inject ->
     check on 512 MiB fp16 tensors (the check_stress command) off-region,
     every submission through counter-and-gate;
  5. ungated: the same with every process registered without gating, so
     nothing excludes the siblings from the timed interval;
  6. frozen (optional): gated, and the holder's regions also stop the
     siblings' process trees and pin the timing thread (CPU exclusivity,
     Section 4.2 steps 4, 5 and 7); frozen_nopin stops them without pinning;
  7. torch_gated / torch_ungated (optional): the siblings are plain torch
     processes looping bf16 4096^3 GEMMs that never call this library; with
     torch_gated they run under the dispatch interceptor (every kernel
     dispatch counted and gated, Section 5), with torch_ungated they run
     unmodified.
t_native is the median of the native run per duration.
"""
import multiprocessing as mp
import os
import sys
import time
import uuid

import numpy as np

from . import stats
from . import workloads as W

MIB = 1 << 20


def _sibling(shm, gated, n, stop, ready, q):
    import torch

    import paper_2609_30057_amd as krex
    torch.cuda.set_device(0)
    cfg = W.CHECK_STRESS
    x = torch.empty(n, dtype=torch.float16, device="cuda:0")
    y = torch.empty_like(x)
    out = krex.check_result_buffer()
    krex.gen(x, cfg["seed"], 0, "uniform", cfg["p0"], cfg["p1"])
    torch.cuda.synchronize()
    krex.attach(0, shm_name=shm, gated=gated)   # registered once initialised (Section 5)
    ready.set()
    rounds = 0
    t0 = time.perf_counter()
    while not stop.is_set():
        krex.gen(x, cfg["seed"], 0, "uniform", cfg["p0"], cfg["p1"])
        krex.inject(y, x, cfg["mask_seed"], cfg["rate"], cfg["delta"], "exact")
        krex.check(y, x, cfg["rtol"], cfg["atol"], out=out)       # reads the verdict: one round in flight
        rounds += 1
    dt = time.perf_counter() - t0
    q.put((rounds, dt, krex.gate_stats()))
    krex.detach()


TORCH_SIBLING = r'''
import os, sys, time
import torch
torch.cuda.set_device(0)
a = torch.randn(4096, 4096, device="cuda", dtype=torch.bfloat16)
b = torch.randn_like(a)
c = a @ b
torch.cuda.synchronize()
print("ready", flush=True)
stop = sys.argv[1]
n = 0
t0 = time.perf_counter()
while not os.path.exists(stop):
    c = a @ b
    torch.cuda.synchronize()
    n += 1
print("rounds %d %.3f" % (n, time.perf_counter() - t0), flush=True)
'''


def _torch_siblings(k, shm, stop_path):
    """k torch GEMM loops; under the dispatch interceptor when shm is given."""
    import subprocess
    from .build import INTERCEPT_LIB
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ)
    env["PYTHONPATH"] = root + os.pathsep + env.get("PYTHONPATH", "")
    if shm:
        env["HSA_TOOLS_LIB"] = INTERCEPT_LIB
        env["KREX_INTERCEPT_SHM"] = shm
    procs = [subprocess.Popen([sys.executable, "-c", TORCH_SIBLING, stop_path], env=env, stdout=subprocess.PIPE,
                              text=True) for _ in range(k)]
    for p in procs:
        if p.stdout.readline().strip() != "ready":
            raise RuntimeError("torch sibling did not start")
    return procs


def _settle(krex, sink, seconds):
    """Back-to-back probe launches for about `seconds`, untimed."""
    import torch
    t0 = time.perf_counter()
    fn = krex.probe_launcher(20000, sink)
    while time.perf_counter() - t0 < seconds:
        krex.time_loop(fn, 0, 20)
    torch.cuda.synchronize()


def _calibrate(krex, sink, target_ms):
    iters = 20000
    for _ in range(4):
        t = float(np.median(krex.time_loop(krex.probe_launcher(iters, sink), 2, 7)))
        iters = max(1, int(round(iters * target_ms / t)))
    t = float(np.median(krex.time_loop(krex.probe_launcher(iters, sink), 2, 7)))
    return iters, t


def _measure(krex, plan, samples, fl, sink, gap_ms, warmup_ms=0.0):
    """warmup_ms > 0: warm-up launches inside the region until about that
    long (so the device's clocks settle after the siblings stop), instead of
    a single one."""
    times, drains = {}, []
    for d, iters in plan:
        fn = krex.probe_launcher(iters, sink)
        warm = max(1, int(round(warmup_ms / d))) if warmup_ms > 0 else 1
        ts = []
        for _ in range(samples):
            ts.append(krex.time_loop(fn, warm, 1, flush_buf=fl, region=True)[0])
            drains.append(krex.gate_stats()["last_drain_ns"] / 1e6)
            time.sleep(gap_ms / 1e3)
        times[d] = ts
    return times, drains


def run(samples=None, durations_ms=None, siblings=None, sibling_elems=None, modes=None, warmup_ms=None,
        settle_s=2.0):
    import torch

    import paper_2609_30057_amd as krex
    cfg = W.SHARED
    samples = samples or cfg["samples"]
    warmup_ms = cfg["warmup_ms"] if warmup_ms is None else warmup_ms
    durations_ms = durations_ms or cfg["probe_ms"]
    siblings = cfg["siblings"] if siblings is None else siblings
    n = sibling_elems or W.CHECK_STRESS["rows"] * W.CHECK_STRESS["cols"]
    torch.cuda.set_device(0)
    fl = torch.empty(cfg["flush_bytes"] // 4, dtype=torch.int32, device="cuda:0")
    sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device="cuda:0")
    ctx = mp.get_context("spawn")
    result = {"metric": "p95 in-region timing inflation (Eq. 1)", "unit": "%", "samples": samples,
              "siblings": siblings, "sibling_workload": "check_stress gen+inject+check, %d fp16 elements" % n,
              "flush_bytes": cfg["flush_bytes"], "gap_ms": cfg["gap_ms"], "P": {}, "P_median_of_10": {},
              "median_ratio": {}, "within_5pct": {}, "calibrated": {}, "sibling_GBps": {}, "drain_ms": {},
              "warmup_ms": warmup_ms}
    times = {}
    modes = list(modes or ("native", "control", "gated", "ungated"))
    compared = [m for m in modes if m != "native"]
    for mode in ["native"] + compared:
        gated = mode not in ("ungated", "torch_ungated")
        shm = "/krex-fid-%s" % uuid.uuid4().hex[:10]
        frozen = mode in ("frozen", "frozen_nopin")
        if mode == "frozen_nopin":
            os.environ["KREX_REGION_CPU"] = "none"
        else:
            os.environ.pop("KREX_REGION_CPU", None)
        krex.attach(0, shm_name=shm, gated=gated, cpu_exclusive=frozen)
        if mode == "native":
            _settle(krex, sink, settle_s)
            plan = []
            for d in durations_ms:
                iters, t = _calibrate(krex, sink, d)
                plan.append((d, iters))
                result["calibrated"][str(d)] = {"iters": iters, "ms": round(t, 4)}
        procs, stop, q = [], ctx.Event(), ctx.Queue()
        torch_procs, stop_path = [], None
        if mode in ("torch_gated", "torch_ungated"):
            stop_path = "/tmp/krex-fid-stop-%s" % uuid.uuid4().hex[:10]
            torch_procs = _torch_siblings(siblings, shm if mode == "torch_gated" else None, stop_path)
        if mode in ("gated", "ungated", "frozen", "frozen_nopin"):
            readies = []
            for _ in range(siblings):
                ready = ctx.Event()
                p = ctx.Process(target=_sibling, args=(shm, gated, n, stop, ready, q))
                p.start()
                procs.append(p)
                readies.append(ready)
            for r in readies:
                if not r.wait(600):
                    raise RuntimeError("sibling did not start")
        t0 = time.perf_counter()
        times[mode], drains = _measure(krex, plan, samples, fl, sink, cfg["gap_ms"], warmup_ms)
        wall = time.perf_counter() - t0
        if torch_procs:
            open(stop_path, "w").close()
            rounds, secs = 0, 0.0
            for p in torch_procs:
                out, _ = p.communicate(timeout=300)
                last = out.strip().splitlines()[-1].split()
                rounds += int(last[1])
                secs = max(secs, float(last[2]))
            os.unlink(stop_path)
            result.setdefault("torch_sibling_TFLOPs", {})[mode] = round(rounds * 2 * 4096**3 / secs / 1e12, 1)
        if procs:
            stop.set()
            got = [q.get(timeout=300) for _ in procs]
            for p in procs:
                p.join(120)
            rounds = sum(g[0] for g in got)
            secs = max(g[1] for g in got)
            result["sibling_GBps"][mode] = round(rounds * 10 * n / secs / 1e9, 1)
            result["sibling_parks"] = result.get("sibling_parks", {})
            result["sibling_parks"][mode] = int(sum(g[2]["parks"] for g in got))
        d = np.asarray(drains)
        result["drain_ms"][mode] = {"p50": round(float(np.median(d)), 4), "p95": round(float(np.percentile(d, 95)), 4),
                                    "max": round(float(d.max()), 4)}
        result.setdefault("wall_s", {})[mode] = round(wall, 1)
        krex.detach()
        print("fidelity: %s done (%.1f s)" % (mode, wall), file=sys.stderr, flush=True)
    for d in durations_ms:
        native = float(np.median(times["native"][d]))
        key = str(d)
        result["P"][key] = {m: round(100 * stats.p95_inflation(times[m][d], native), 3)
                            for m in compared}
        nat10 = float(np.median(stats.medians_of(times["native"][d])))
        result["P_median_of_10"][key] = {m: round(100 * stats.p95_inflation(stats.medians_of(times[m][d]), nat10), 3)
                                         for m in compared}
        result["median_ratio"][key] = {m: round(stats.median_ratio(times[m][d], native), 4)
                                       for m in compared}
        result["within_5pct"][key] = {m: round(stats.within(times[m][d], native), 4)
                                      for m in compared}
        result["calibrated"][key]["native_median_ms"] = round(native, 4)
        result.setdefault("ratio_quantiles", {})[key] = {
            m: [round(float(q), 4) for q in np.percentile(np.asarray(times[m][d]) / native, [5, 50, 90, 95, 99, 100])]
            for m in ["native"] + compared}
    return result
