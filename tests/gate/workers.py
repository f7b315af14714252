"""Process bodies for the region-coordinator tests (spawned, so each has its
own copy of the coordinator's process state)."""
import ctypes
import time

from tests.gate import harness

OK = 0


def _L(variant=""):
    return harness.load(variant)


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
