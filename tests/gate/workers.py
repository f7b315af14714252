"""Process bodies for the region-coordinator tests (spawned, so each has its
own copy of the coordinator's process state)."""
import ctypes
import os
import time

from tests.gate import harness

OK = 0


def _L(variant=""):
    # KREX_GATE_VARIANT selects the build for every worker of a test run
    # (the ThreadSanitizer variant is loaded under libtsan, preloaded by the
    # test that spawns these processes)
    return harness.load(variant or os.environ.get("KREX_GATE_VARIANT", ""))


def sibling_loop(name, dur_us, seconds, depth, q, variant=""):
    L = _L(variant)
    assert L.kg_attach(name.encode(), 0) == OK
    end = time.monotonic() + seconds
    n = 0
    while time.monotonic() < end:
        if L.kg_inflight() < depth:
            rc = L.kg_submit(dur_us, 0, None)
            assert rc == OK, rc
            n += 1
        else:
            time.sleep(dur_us * 1e-6 / 4)
    L.kg_wait_idle(60000)
    q.put(("sibling", harness.log(L), harness.stats(L)))
    L.kg_detach()


def holder_loop(name, regions, region_ms, gap_ms, start_delay, q, variant=""):
    L = _L(variant)
    assert L.kg_attach(name.encode(), 0) == OK
    time.sleep(start_delay)
    windows = []
    for _ in range(regions):
        rc = L.kg_region_begin(10000)
        assert rc == OK, rc
        t_in = L.kg_now()
        time.sleep(region_ms / 1000)
        t_out = L.kg_now()
        assert L.kg_region_end() == OK
        windows.append((t_in, t_out))
        time.sleep(gap_ms / 1000)
    q.put(("holder", windows, harness.stats(L)))
    L.kg_detach()


def hold_region(name, hold_s, ready, q):
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    assert L.kg_region_begin(10000) == OK
    ready.set()
    time.sleep(hold_s)
    t_end = L.kg_now()
    assert L.kg_region_end() == OK
    q.put(("held", t_end))
    L.kg_detach()


def hold_and_die(name, ready):
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    assert L.kg_region_begin(10000) == OK
    ready.set()
    time.sleep(600)


def long_op_then_sleep(name, dur_us, ready):
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    assert L.kg_submit(dur_us, 0, None) == OK
    ready.set()
    time.sleep(600)


def try_region(name, timeout_ms, q):
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    t0 = time.monotonic()
    rc = L.kg_region_begin(timeout_ms)
    dt = time.monotonic() - t0
    if rc >= 0:
        L.kg_region_end()
    q.put(("try", rc, dt, harness.stats(L)))
    L.kg_detach()


def submit_once(name, flags, timeout_ns, q):
    L = _L()
    assert L.kg_attach(name.encode(), flags) == OK
    t0 = L.kg_now()
    t = ctypes.c_uint64()
    rc = L.kg_submit(100, timeout_ns, ctypes.byref(t))
    L.kg_wait_idle(10000)
    q.put(("submit", rc, t0, t.value, harness.stats(L)))
    L.kg_detach()


def spinner(name, counter, child_counter, ready, stop):
    """Registered process that spins on the CPU, with a forked child that
    spins too (a process tree of two)."""
    import os
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    pid = os.fork()
    if pid == 0:
        while not stop.is_set():
            child_counter.value += 1
        os._exit(0)
    ready.set()
    while not stop.is_set():
        counter.value += 1
    os.waitpid(pid, 0)
    L.kg_detach()


def exclusive_holder(name, counters, regions, region_ms, q):
    """Holder with CPU exclusivity: samples the siblings' counters inside and
    after each region, and its own affinity inside and after."""
    import os
    L = _L()
    assert L.kg_attach(name.encode(), 2) == OK
    before = len(os.sched_getaffinity(0))
    res = []
    for _ in range(regions):
        assert L.kg_region_begin(10000) == OK
        aff_in = len(os.sched_getaffinity(0))
        c0 = [c.value for c in counters]
        time.sleep(region_ms / 1000)
        c1 = [c.value for c in counters]
        frozen = harness.stats(L)["last_frozen"]
        assert L.kg_region_end() == OK
        aff_out = len(os.sched_getaffinity(0))
        time.sleep(0.05)
        c2 = [c.value for c in counters]
        res.append((c0, c1, c2, aff_in, aff_out, frozen))
    q.put(("excl", before, res))
    L.kg_detach()


def exclusive_hold_and_die(name, ready):
    L = _L()
    assert L.kg_attach(name.encode(), 2) == OK
    assert L.kg_region_begin(10000) == OK
    ready.set()
    time.sleep(600)


def registered_parent_of_holder(name, counter, q):
    """A registered process whose child is an exclusive holder: the holder
    must not stop itself while stopping its parent's tree."""
    import multiprocessing as mp
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    ctx = mp.get_context("spawn")
    cq = ctx.Queue()
    child = ctx.Process(target=exclusive_holder, args=(name, [counter], 2, 100, cq))
    child.start()
    got = cq.get(timeout=60)
    child.join(60)
    q.put(("parent", child.exitcode, got))
    L.kg_detach()


def long_op_then_fail(name, dur_us, ready):
    """Submits one long operation, then fails its health check (its work
    would still be in flight) and stays alive."""
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    assert L.kg_submit(dur_us, 0, None) == OK
    L.kg_fail()
    ready.set()
    time.sleep(600)


def fail_then_submit(name, q):
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    assert L.kg_submit(100, 0, None) == OK
    L.kg_wait_idle(10000)
    L.kg_fail()
    rc = L.kg_submit(100, 0, None)
    q.put(("failed_submit", rc))
    L.kg_detach()


def hold_past_lease(name, hold_s, second_ms, ready, ready2, q):
    """Holds a region for hold_s (beyond the lease), then a short second one
    (within it), signalling ready2 once inside the second."""
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    assert L.kg_region_begin(10000) == OK
    t_in = L.kg_now()
    ready.set()
    time.sleep(hold_s)
    rc1 = L.kg_region_end()
    assert L.kg_region_begin(10000) == OK
    t2_in = L.kg_now()
    ready2.set()
    time.sleep(second_ms / 1000)
    t2_out = L.kg_now()
    rc2 = L.kg_region_end()
    q.put(("holder", rc1, rc2, t_in, t2_in, t2_out))
    L.kg_detach()


def submit_twice(name, ready2, q):
    """Two submissions: the first parks until the first region is revoked,
    the second is made inside the holder's short second region."""
    L = _L()
    assert L.kg_attach(name.encode(), 0) == OK
    t = ctypes.c_uint64()
    rc = L.kg_submit(100, 10**10, ctypes.byref(t))
    t1 = t.value
    assert ready2.wait(30)
    rc2 = L.kg_submit(100, 10**10, ctypes.byref(t))
    t2 = t.value
    L.kg_wait_idle(10000)
    q.put(("sib", rc, t1, rc2, t2, harness.stats(L)))
    L.kg_detach()


def report_loaded(q):
    """Which coordinator build and sanitizer runtime this process mapped."""
    _L()
    with open("/proc/self/maps") as f:
        maps = f.read()
    q.put(("loaded", "libtsan" in maps, "libgate_harness_tsan.so" in maps))
