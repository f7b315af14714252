"""GPU flush, probe, fixture GEMM, timed loop and critical regions.

Flush content and eviction (a re-read right after a flush larger than the
Infinity Cache runs at HBM speed rather than cache speed); the probe and the
naive GEMM bit for bit against the oracle; the timed loop's event timings of
a known-duration kernel; region entry / exit states; and two processes on
one GPU generating and checking under a held region with results identical
to a solo run (Section 2.1: colocated work does not change generated tensors
or verdicts)."""
import multiprocessing as mp
import os
import time
import uuid

import numpy as np
import pytest
import torch

import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import assert_bits_equal, empty, from_storage, same_result, to_storage

pytestmark = pytest.mark.gpu


@pytest.fixture
def shm_name():
    name = "/krex-gtest-%s" % uuid.uuid4().hex[:12]
    yield name
    try:
        os.unlink("/dev/shm" + name)
    except FileNotFoundError:
        pass


def test_flush_content():
    for nbytes in (16, 4096 + 16, (64 << 20) + 48):
        buf = torch.zeros(nbytes // 4, dtype=torch.int32, device="cuda")
        krex.flush(buf, 0xA5A5F00D)
        got = buf.cpu().numpy().view(np.uint32)
        ref = np.zeros(nbytes // 4, dtype=np.uint32)
        oracle.flush_fill(ref, 0xA5A5F00D)
        assert np.array_equal(got, ref)
    with pytest.raises(krex.KrexError):
        krex.flush(torch.zeros(5, dtype=torch.int32, device="cuda"), 1)


def test_flush_evicts_cached_data():
    """A 64 MiB buffer read right after a 1 GiB flush must read at the cold
    HBM rate: no faster than 0.9 x the time of a cold read of the same size
    (a 64 MiB slice of a 2 GiB buffer, written in order and read in order, so
    at least 1.3 GiB of other traffic separates each slice's last touch from
    its read), while a re-read without the flush is clearly faster (the
    buffer fits in the 256 MB Infinity Cache), so the test can tell the
    states apart. A flush that evicted only part of the buffer would put the
    flushed read between the two."""
    x = torch.ones(16 << 20, dtype=torch.float32, device="cuda")
    fl = torch.empty(1 << 28, dtype=torch.int32, device="cuda")
    W = torch.empty(32, 16 << 20, dtype=torch.float32, device="cuda")
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed_read(t):
        s.record()
        t.sum()
        e.record()
        torch.cuda.synchronize()
        return s.elapsed_time(e)

    for _ in range(5):            # the reduction's one-time setup stays out of the samples
        timed_read(x)
    warm, flushed = [], []
    for _ in range(11):
        x.sum()
        warm.append(timed_read(x))
        krex.flush(fl, 7)
        flushed.append(timed_read(x))
    W.fill_(1.0)
    cold = [timed_read(W[k]) for k in range(11)]
    w, f, c = np.median(warm), np.median(flushed), np.median(cold)
    assert f >= 0.9 * c, ("flushed read faster than a cold one", warm, flushed, cold)
    assert w <= 0.85 * c, ("a re-read is not faster than a cold read: the test cannot see the cache", warm, cold)


def test_probe_matches_oracle():
    sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device="cuda")
    for iters in (0, 1, 37, 500):
        krex.probe(iters, sink)
        assert_bits_equal(sink.cpu().numpy(), oracle.probe(iters), "probe %d" % iters)


def test_probe_clock_record():
    """The clocked probe writes the same sink and a sane clock record per
    wave: cycles and real-time ticks both advance, the implied shader clock
    lies between 0.5 and 3 GHz, and every wave's interval sits inside the
    kernel's event-timed interval."""
    import numpy as np
    sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device="cuda")
    clocks = torch.zeros(krex.PROBE_WAVES * krex.PROBE_CLOCK_WORDS, dtype=torch.int64, device="cuda")
    krex.probe(500, sink, clocks=clocks)
    assert_bits_equal(sink.cpu().numpy(), oracle.probe(500), "clocked probe 500")
    iters = 30000
    times = krex.time_loop(krex.probe_launcher(iters, sink, clocks), 2, 1)
    c = krex.probe_clocks(clocks)
    assert np.all(c["cycles"] > 0) and np.all(c["rt_ticks"] > 0)
    assert np.all((c["mhz"] > 500) & (c["mhz"] < 3000)), (c["mhz"].min(), c["mhz"].max())
    span_ms = (c["rt_end"].max() - c["rt_start"].min()) / 1e5
    assert 0.5 * times[0] < span_ms <= times[0] * 1.02 + 0.01, (span_ms, times)
    print("probe clocks: MHz p5/p50/p95 %s, XCC_ID values %s, distinct HW_ID %d" % (
        np.percentile(c["mhz"], [5, 50, 95]).round(1), np.unique(c["xcc"]), np.unique(c["hw_id"]).size), flush=True)
    assert np.all((c["xcc"] >= 0) & (c["xcc"] < 16))
    assert_bits_equal(sink.cpu().numpy(), oracle.probe(iters), "clocked probe in the loop")


def test_fixture_sgemm_matches_oracle():
    A = empty("f32", 256 * 256)
    B = empty("f32", 256 * 256)
    krex.gen(A, 0, 0)
    krex.gen(B, 0, 65536)
    C = torch.empty(256, 256, dtype=torch.float32, device="cuda")
    krex.fixture_sgemm(A.view(256, 256), B.view(256, 256), C)
    Ar = oracle.gen("f32", 65536, 0, 0).reshape(256, 256)
    Br = oracle.gen("f32", 65536, 0, 65536).reshape(256, 256)
    assert_bits_equal(C.cpu().numpy(), oracle.sgemm(Ar, Br), "sgemm")


def test_time_loop_known_duration():
    sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device="cuda")
    fn = krex.probe_launcher(20000, sink)
    t1 = krex.time_loop(fn, 2, 10)
    fn2 = krex.probe_launcher(40000, sink)
    t2 = krex.time_loop(fn2, 2, 10)
    m1, m2 = np.median(t1), np.median(t2)
    assert all(t > 0 for t in t1 + t2)
    assert 1.7 < m2 / m1 < 2.3, (m1, m2)


def test_time_loop_flush_times_and_python_callable():
    fl = torch.empty(1 << 28, dtype=torch.int32, device="cuda")   # 1 GiB
    a = torch.randn(2048, 2048, device="cuda")
    b = torch.randn(2048, 2048, device="cuda")
    c = torch.empty(2048, 2048, device="cuda")
    times, ftimes = krex.time_loop(lambda: torch.matmul(a, b, out=c), 3, 5, flush_buf=fl, with_flush_times=True)
    assert len(times) == 5 and all(t > 0 for t in times)
    gbps = [(1 << 30) / (ft * 1e-3) / 1e9 for ft in ftimes]
    assert all(1000 < g < 9000 for g in gbps), gbps
    assert (fl.view(torch.int32)[:4].cpu().numpy().view(np.uint32) == np.uint32(0x9E3779B9 * 5 & 0xFFFFFFFF)).all()


def test_region_states(shm_name):
    with pytest.raises(krex.KrexError) as e:
        krex.region_begin()
    assert e.value.status == krex.ENOTATTACHED
    krex.attach(shm_name=shm_name)
    try:
        st = krex.gate_stats()
        assert st["slot"] >= 0 and st["gated"] == 1
        fl = torch.empty(1 << 27, dtype=torch.int32, device="cuda")
        with krex.region.critical(flush_buf=fl):
            with pytest.raises(krex.KrexError) as e:
                krex.region_begin()
            assert e.value.status == krex.ESTATE
            x = empty("f16", 1 << 20)
            krex.gen(x, 1)                       # the holder's own submissions pass its gate
        sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device="cuda")
        t = krex.time_loop(krex.probe_launcher(1000, sink), 1, 5, flush_buf=fl, region=True)
        assert len(t) == 5
        assert krex.gate_stats()["regions"] == 2
        with pytest.raises(krex.KrexError):
            krex.region_end()
    finally:
        krex.detach()


def _sibling(shm_name, q, seconds, ready):
    import torch as th
    import paper_2609_30057_amd as k
    th.cuda.init()
    n = 1 << 24
    x = th.empty(n, dtype=th.float16, device="cuda")
    y = th.empty_like(x)
    out = k.check_result_buffer()
    k.gen(x, 2, 0, "uniform", -4.0, 4.0)
    th.cuda.synchronize()
    k.attach(shm_name=shm_name)                  # registered once initialised (stopped only after this)
    ready.set()
    end = time.monotonic() + seconds
    results = set()
    rounds = 0
    while time.monotonic() < end:
        k.gen(x, 2, 0, "uniform", -4.0, 4.0)
        k.inject(y, x, 3, 0.001, 0.5, "exact")
        r = k.check(y, x, 1e-3, 1e-3, out=out)
        results.add((r.mismatches, r.argmax_abs, r.max_abs, r.max_rel, int(x[12345].view(th.int16))))
        rounds += 1
    q.put((sorted(results), rounds, k.gate_stats()))
    k.detach()


@pytest.mark.parametrize("cpu_exclusive", [False, True], ids=["gated", "cpu_exclusive"])
def test_two_processes_share_gpu_invariant_results(shm_name, cpu_exclusive):
    """A sibling loops gen -> inject -> check while this process holds
    regions (with CPU exclusivity: the sibling is stopped inside them); every
    sibling round gives the solo result."""
    n = 1 << 24
    x = torch.empty(n, dtype=torch.float16, device="cuda")
    y = torch.empty_like(x)
    krex.gen(x, 2, 0, "uniform", -4.0, 4.0)
    krex.inject(y, x, 3, 0.001, 0.5, "exact")
    solo = krex.check(y, x, 1e-3, 1e-3)
    solo_key = (solo.mismatches, solo.argmax_abs, solo.max_abs, solo.max_rel, int(x[12345].view(torch.int16)))
    ctx = mp.get_context("spawn")
    q = ctx.Queue()
    ready = ctx.Event()
    p = ctx.Process(target=_sibling, args=(shm_name, q, 4.0, ready))
    p.start()
    krex.attach(shm_name=shm_name, cpu_exclusive=cpu_exclusive)
    frozen = []
    try:
        sink = torch.empty(krex.PROBE_THREADS, dtype=torch.float32, device="cuda")
        assert ready.wait(120)
        time.sleep(0.3)
        for _ in range(10):
            krex.time_loop(krex.probe_launcher(20000, sink), 1, 3, region=True)
            frozen.append(krex.gate_stats()["last_frozen"])
            time.sleep(0.05)
        drains = krex.gate_stats()
    finally:
        results, rounds, st = q.get(timeout=120)
        p.join(60)
        krex.detach()
    assert p.exitcode == 0
    assert rounds > 3 and results == [solo_key]
    assert drains["regions"] == 10
    assert frozen == ([1] * 10 if cpu_exclusive else [0] * 10)


def test_health_check(shm_name):
    """Section 4.3: a healthy context passes; a stream left in graph capture
    fails the check, which retires the process's slot (further submissions
    are refused)."""
    krex.attach(shm_name=shm_name)
    try:
        x = empty("f16", 1 << 20)
        krex.gen(x, 1)
        assert krex.health_check() == krex.OK
        s = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        y = torch.zeros(16, device="cuda")
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.capture_begin()
            try:
                y.add_(1.0)
                with pytest.raises(krex.KrexError) as e:
                    krex.health_check(stream=s)
                assert e.value.status == krex.ESTATE
            finally:
                g.capture_end()
        torch.cuda.synchronize()
        with pytest.raises(krex.KrexError) as e:
            krex.gen(x, 1)
        assert e.value.status == krex.EHIP
    finally:
        krex.detach()
    krex.attach(shm_name=shm_name)                # a new registration starts healthy
    try:
        krex.gen(x, 1)
        assert krex.health_check() == krex.OK
    finally:
        krex.detach()
