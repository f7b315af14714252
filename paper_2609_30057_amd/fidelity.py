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
  1. calibrate the probe's iteration count to each target duration, alone,
     and record the slowest wave's clock of those launches;
  2. native: `samples` single-shot timings per duration, alone (each sample:
     region entry, warm-up, a 512 MiB flush, one timed launch, exit; then a
     5 ms off-region gap). The warm-up launches the probe one launch at a
     time until its slowest wave runs at the calibration clock, at most 20
     ms (warmup="clock", the default), or for about warmup_ms (warmup="time";
     exactly one launch with warmup_ms = 0). Every timed launch records its
     waves' clocks: its duration is their fixed cycle count over the slowest
     wave's clock plus a constant launch overhead, so the clock records
     account for every sample's time;
  3. control: the same again (native repeat);
  4. gated: the same while `siblings` processes loop generate -> inject ->
     check on 512 MiB fp16 tensors (the check_stress command) off-region,
     every submission through counter-and-gate;
  5. ungated: the same with every process registered without gating, so
     nothing excludes the siblings from the timed interval;
  5b. gated_chunked (optional): gated, with the siblings splitting their
     generation and injection into separately admitted 64 MiB launches, at
     most two in flight (KREX_CHUNK_BYTES), so a region's drain waits for
     less sibling work;
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


def _sibling(shm, gated, n, stop, ready, q, chunk_bytes=0):
    if chunk_bytes:
        # read by the library at its first chunkable call in this process
        os.environ["KREX_CHUNK_BYTES"] = str(chunk_bytes)
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
    """Iterations for a probe of about target_ms alone; returns (iters, median
    ms, median over the last calibration launches of each launch's slowest
    wave clock in MHz)."""
    import torch
    iters = 20000
    for _ in range(4):
        t = float(np.median(krex.time_loop(krex.probe_launcher(iters, sink), 2, 7)))
        iters = max(1, int(round(iters * target_ms / t)))
    clk = torch.zeros(krex.PROBE_WAVES * krex.PROBE_CLOCK_WORDS, dtype=torch.int64, device="cuda:0")
    ts, mhz = [], []
    for _ in range(7):
        ts.append(krex.time_loop(krex.probe_launcher(iters, sink, clk), 2, 1)[0])
        mhz.append(float(np.nanmin(krex.probe_clocks(clk)["mhz"])))
    return iters, float(np.median(ts)), float(np.median(mhz))


def clock_summary(clk):
    """Per-sample clock figures from a (samples, PROBE_WAVES * 8) int64 tensor
    of probe clock records: the median and minimum of the waves' effective
    shader clocks (MHz), and the real-time span of the launch (first wave
    start to last wave end, ms)."""
    a = clk.cpu().numpy().view(np.uint64).reshape(clk.shape[0], -1, 8)
    cyc = (a[:, :, 1] - a[:, :, 0]).astype(np.float64)
    rt = (a[:, :, 3] - a[:, :, 2]).astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        mhz = np.where(rt > 0, cyc / rt * 100.0, np.nan)
    span = (a[:, :, 3].max(axis=1) - a[:, :, 2].min(axis=1)).astype(np.float64) / 1e5
    start_skew = (a[:, :, 2].max(axis=1) - a[:, :, 2].min(axis=1)).astype(np.float64) / 1e5
    return {"mhz_med": np.nanmedian(mhz, axis=1), "mhz_min": np.nanmin(mhz, axis=1), "span_ms": span,
            "start_skew_ms": start_skew, "wave_ms_max": rt.max(axis=1) / 1e5,
            "wave_cycles_med": np.median(cyc, axis=1), "wave_cycles_max": cyc.max(axis=1)}


def _measure(krex, plan, samples, fl, sink, gap_ms, warmup_ms=0.0, warm_clock=None):
    """Single-shot samples of each (duration, iters) of `plan`, each in its
    own region. warmup_ms > 0: warm-up launches inside the region for about
    that long before the flush and the timed launch (so the device's clocks
    settle after the siblings stop); 0: one warm-up launch. warm_clock =
    (target_mhz, cap_ms, lead): instead, warm-up launches one at a time, each
    followed by a read of its clock record, until the slowest wave's clock
    reaches target_mhz (at least one launch; stop after cap_ms; the slowest
    wave counts, since the launch lasts as long as it does), then `lead`
    more launches enqueued without a wait right before the flush and the
    timed launch. Every timed launch records its clocks. Returns times,
    drains, clock summaries and warm-up launch counts per duration."""
    import torch
    times, drains, clocks, warms = {}, [], {}, {}
    words = krex.PROBE_WAVES * krex.PROBE_CLOCK_WORDS
    for d, iters in plan:
        clk = torch.zeros((samples, words), dtype=torch.int64, device="cuda:0")
        wclk = torch.zeros(words, dtype=torch.int64, device="cuda:0")
        warm = max(1, int(round(warmup_ms / d))) if warmup_ms > 0 else 1
        wfn = krex.probe_launcher(iters, sink, wclk)
        ts, nw = [], []
        for i in range(samples):
            fn = krex.probe_launcher(iters, sink, clk[i])
            if warm_clock is None:
                ts.append(krex.time_loop(fn, warm, 1, flush_buf=fl, region=True)[0])
                nw.append(warm)
            else:
                target, cap_ms, lead = warm_clock
                krex.region_begin()
                try:
                    n, t0 = 0, time.perf_counter()
                    while True:
                        krex.time_loop(wfn, 0, 1)          # one launch, synchronised
                        n += 1
                        mhz = float(np.nanmin(krex.probe_clocks(wclk)["mhz"]))
                        if mhz >= target or (time.perf_counter() - t0) * 1e3 >= cap_ms:
                            break
                    # lead: launches enqueued right before the flush and the
                    # timed launch, so the device does not idle between them
                    for _ in range(lead):
                        krex.probe(iters, sink)
                    ts.append(krex.time_loop(fn, 0, 1, flush_buf=fl)[0])
                finally:
                    krex.region_end()
                nw.append(n)
            drains.append(krex.gate_stats()["last_drain_ns"] / 1e6)
            time.sleep(gap_ms / 1e3)
        times[d] = ts
        clocks[d] = clock_summary(clk)
        warms[d] = nw
        del clk
    return times, drains, clocks, warms


def run(samples=None, durations_ms=None, siblings=None, sibling_elems=None, modes=None, warmup_ms=None,
        settle_s=2.0, warmup=None, sessions=1, clock_cap_ms=None, dump=None, lead=None):
    """warmup: "time" (launches for about warmup_ms in each region) or
    "clock" (launches until the slowest wave's clock reaches the calibration
    median, at most clock_cap_ms), the same procedure for every mode, the
    native run included. sessions: how many times the compared modes are
    measured in turn after the native run (P per session in P_sessions; P is
    the first session's). dump: a path for an .npz of every sample's time
    and clock figures."""
    import torch

    import paper_2609_30057_amd as krex
    cfg = W.SHARED
    samples = samples or cfg["samples"]
    warmup_ms = cfg["warmup_ms"] if warmup_ms is None else warmup_ms
    warmup = cfg["warmup"] if warmup is None else warmup
    clock_cap_ms = cfg["clock_cap_ms"] if clock_cap_ms is None else clock_cap_ms
    lead = cfg.get("lead", 0) if lead is None else lead
    durations_ms = durations_ms or cfg["probe_ms"]
    siblings = cfg["siblings"] if siblings is None else siblings
    n = sibling_elems or W.CHECK_STRESS["rows"] * W.CHECK_STRESS["cols"]
    if warmup not in ("time", "clock"):
        raise ValueError("warmup is 'time' or 'clock'")
    torch.cuda.set_device(0)
    fl = torch.empty(cfg["flush_bytes"] // 4, dtype=torch.int32, device="cuda:0")
    sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device="cuda:0")
    ctx = mp.get_context("spawn")
    result = {"metric": "p95 in-region timing inflation (Eq. 1)", "unit": "%", "samples": samples,
              "siblings": siblings, "sibling_workload": "check_stress gen+inject+check, %d fp16 elements" % n,
              "flush_bytes": cfg["flush_bytes"], "gap_ms": cfg["gap_ms"], "P": {}, "P_median_of_10": {},
              "median_ratio": {}, "within_5pct": {}, "calibrated": {}, "sibling_GBps": {}, "drain_ms": {},
              "warmup": warmup, "warmup_ms": warmup_ms if warmup == "time" else None,
              "clock_cap_ms": clock_cap_ms if warmup == "clock" else None,
              "lead": lead if warmup == "clock" else None, "sessions": sessions}
    times, clocks, warms = {}, {}, {}
    modes = list(modes or ("native", "control", "gated", "ungated"))
    compared = [m for m in modes if m != "native"]
    runs = [("native", 0)] + [(m, k) for k in range(sessions) for m in compared]
    plan, targets = [], {}
    for mode, sess in runs:
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
            for d in durations_ms:
                iters, t, mhz = _calibrate(krex, sink, d)
                plan.append((d, iters))
                targets[d] = mhz
                result["calibrated"][str(d)] = {"iters": iters, "ms": round(t, 4), "clock_MHz": round(mhz, 1)}
        procs, stop, q = [], ctx.Event(), ctx.Queue()
        torch_procs, stop_path = [], None
        if mode in ("torch_gated", "torch_ungated"):
            stop_path = "/tmp/krex-fid-stop-%s" % uuid.uuid4().hex[:10]
            torch_procs = _torch_siblings(siblings, shm if mode == "torch_gated" else None, stop_path)
        if mode in ("gated", "ungated", "frozen", "frozen_nopin", "gated_chunked"):
            readies = []
            chunk = cfg["chunk_bytes"] if mode == "gated_chunked" else 0
            for _ in range(siblings):
                ready = ctx.Event()
                p = ctx.Process(target=_sibling, args=(shm, gated, n, stop, ready, q, chunk))
                p.start()
                procs.append(p)
                readies.append(ready)
            for r in readies:
                if not r.wait(600):
                    raise RuntimeError("sibling did not start")
        t0 = time.perf_counter()
        key = (mode, sess)
        tm, drains, ck, wm = {}, [], {}, {}
        for d, iters in plan:
            wc = (targets[d], clock_cap_ms, lead) if warmup == "clock" else None
            a, b, c, e = _measure(krex, [(d, iters)], samples, fl, sink, cfg["gap_ms"], warmup_ms, wc)
            tm.update(a)
            drains += b
            ck.update(c)
            wm.update(e)
        times[key], clocks[key], warms[key] = tm, ck, wm
        wall = time.perf_counter() - t0
        tag = mode if sess == 0 else "%s#%d" % (mode, sess)
        if torch_procs:
            open(stop_path, "w").close()
            rounds, secs = 0, 0.0
            for p in torch_procs:
                out, _ = p.communicate(timeout=300)
                last = out.strip().splitlines()[-1].split()
                rounds += int(last[1])
                secs = max(secs, float(last[2]))
            os.unlink(stop_path)
            result.setdefault("torch_sibling_TFLOPs", {})[tag] = round(rounds * 2 * 4096**3 / secs / 1e12, 1)
        if procs:
            stop.set()
            got = [q.get(timeout=300) for _ in procs]
            for p in procs:
                p.join(120)
            rounds = sum(g[0] for g in got)
            secs = max(g[1] for g in got)
            result["sibling_GBps"][tag] = round(rounds * 10 * n / secs / 1e9, 1)
            result.setdefault("sibling_parks", {})[tag] = int(sum(g[2]["parks"] for g in got))
        dd = np.asarray(drains)
        result["drain_ms"][tag] = {"p50": round(float(np.median(dd)), 4), "p95": round(float(np.percentile(dd, 95)), 4),
                                   "max": round(float(dd.max()), 4)}
        result.setdefault("wall_s", {})[tag] = round(wall, 1)
        krex.detach()
        print("fidelity: %s done (%.1f s)" % (tag, wall), file=sys.stderr, flush=True)
    nat = ("native", 0)
    for d in durations_ms:
        native = float(np.median(times[nat][d]))
        nat_mhz = float(np.median(clocks[nat][d]["mhz_med"]))
        key = str(d)
        first = {m: (m, 0) for m in compared}
        result["P"][key] = {m: round(100 * stats.p95_inflation(times[k][d], native), 3) for m, k in first.items()}
        if sessions > 1:
            result.setdefault("P_sessions", {})[key] = {
                m: [round(100 * stats.p95_inflation(times[(m, s)][d], native), 3) for s in range(sessions)]
                for m in compared}
        nat10 = float(np.median(stats.medians_of(times[nat][d])))
        result["P_median_of_10"][key] = {m: round(100 * stats.p95_inflation(stats.medians_of(times[k][d]), nat10), 3)
                                         for m, k in first.items()}
        result["median_ratio"][key] = {m: round(stats.median_ratio(times[k][d], native), 4)
                                       for m, k in first.items()}
        result["within_5pct"][key] = {m: round(stats.within(times[k][d], native), 4) for m, k in first.items()}
        result["calibrated"][key]["native_median_ms"] = round(native, 4)
        result.setdefault("ratio_quantiles", {})[key] = {
            m: [round(float(q), 4) for q in np.percentile(np.asarray(times[k][d]) / native, [5, 50, 90, 95, 99, 100])]
            for m, k in [("native", nat)] + list(first.items())}
        # Clock evidence per sample: each timed launch's median wave clock.
        # clock_corrected: the sample's time scaled to the native run's
        # median clock (t f / f_native), i.e. what is left once the clock
        # difference is taken out.
        cl = {}
        for m, k in [("native", nat)] + list(first.items()):
            t = np.asarray(times[k][d])
            f = clocks[k][d]["mhz_med"]
            r = t / native
            ok = np.isfinite(f)
            corr = float(np.corrcoef(r[ok], nat_mhz / f[ok])[0, 1]) if ok.sum() > 2 and np.std(f[ok]) > 0 else None
            ck = clocks[k][d]
            # where the time goes, medians over the samples: the event-timed
            # launch = (event overhead) + (first wave start .. last wave end);
            # that span = (start skew of the waves) + (the rest, at most the
            # longest wave)
            cl[m + "_decomposition_us"] = {
                "event": round(float(np.median(t)) * 1e3, 2),
                "event_minus_span": round(float(np.median(t - ck["span_ms"])) * 1e3, 2),
                "span": round(float(np.median(ck["span_ms"])) * 1e3, 2),
                "start_skew": round(float(np.median(ck["start_skew_ms"])) * 1e3, 2),
                "longest_wave": round(float(np.median(ck["wave_ms_max"])) * 1e3, 2),
                "wave_cycles_median": int(np.median(ck["wave_cycles_med"])),
                "wave_cycles_max": int(np.median(ck["wave_cycles_max"]))}
            cl[m] = {"MHz_p5_p50_p95": [round(float(v), 1) for v in np.nanpercentile(f, [5, 50, 95])],
                     "MHz_min_wave_p5": round(float(np.nanpercentile(clocks[k][d]["mhz_min"], 5)), 1),
                     "corr_ratio_vs_clock_deficit": None if corr is None else round(corr, 3),
                     "P_clock_corrected": round(100 * stats.p95_inflation(t[ok] * f[ok] / nat_mhz, native), 3),
                     "warmup_launches_p50_p95": [int(np.median(warms[k][d])),
                                                 int(np.percentile(warms[k][d], 95))]}
        result.setdefault("clock", {})[key] = cl
    if dump:
        arrays = {}
        for (mode, sess), per in times.items():
            for d, ts in per.items():
                tag = "%s_%d_%g" % (mode, sess, d)
                arrays["t_" + tag] = np.asarray(ts)
                for name, v in clocks[(mode, sess)][d].items():
                    arrays[name + "_" + tag] = np.asarray(v)
        np.savez_compressed(dump, **arrays)
    return result
