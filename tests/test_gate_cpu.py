"""Region coordinator (csrc/gate.cpp) driven by several processes over a fake
in-order device, on the CPU. Checks the protocol of Section 4.2: region lock,
gate with holder and epoch, drain of siblings' in-flight work, parking of
submissions while the gate is closed, entry failure leaving nothing held,
and recovery from dead holders and dead siblings; plus Section 5's
completion-counter variant (counts released when operations finish)."""
import multiprocessing as mp
import os
import signal
import time
import uuid

import pytest

from tests.gate import harness, workers

CTX = mp.get_context("spawn")
OK, RECOVERED, ETIMEDOUT, ESTATE, ENOTATTACHED, EPEER = 0, 1, -4, -5, -6, -8


@pytest.fixture
def shm_name():
    name = "/krex-test-%s" % uuid.uuid4().hex[:12]
    yield name
    try:
        os.unlink("/dev/shm" + name)
    except FileNotFoundError:
        pass


@pytest.fixture(scope="module", autouse=True)
def built():
    harness.build()


def _collect(q, n, timeout=60):
    out = []
    for _ in range(n):
        out.append(q.get(timeout=timeout))
    return out


def _join(procs, timeout=60):
    for p in procs:
        p.join(timeout)
        assert p.exitcode == 0, (p.name, p.exitcode)


def test_no_sibling_work_runs_inside_regions(shm_name):
    """Every sibling operation executes entirely outside every region window
    [entered, exit requested] of the holder."""
    q = CTX.Queue()
    sibs = [CTX.Process(target=workers.sibling_loop, args=(shm_name, 3000, 2.5, 3, q)) for _ in range(3)]
    holder = CTX.Process(target=workers.holder_loop, args=(shm_name, 8, 40, 60, 0.5, q))
    for p in sibs + [holder]:
        p.start()
    res = _collect(q, 4)
    _join(sibs + [holder])
    windows = [r for r in res if r[0] == "holder"][0][1]
    ops = [op for r in res if r[0] == "sibling" for op in r[1]]
    assert len(windows) == 8 and len(ops) > 200
    for (s, e) in ops:
        for (a, b) in windows:
            assert e <= a or s >= b, "sibling op [%d, %d] overlaps region [%d, %d]" % (s, e, a, b)
    sib_stats = [r[2] for r in res if r[0] == "sibling"]
    assert sum(s["parks"] for s in sib_stats) > 0          # siblings did meet the closed gate


def test_entry_times_out_while_another_holds(shm_name):
    q = CTX.Queue()
    ready = CTX.Event()
    a = CTX.Process(target=workers.hold_region, args=(shm_name, 1.5, ready, q))
    a.start()
    assert ready.wait(30)
    b = CTX.Process(target=workers.try_region, args=(shm_name, 200, q))
    b.start()
    tag, rc, dt, _ = q.get(timeout=30)
    assert tag == "try" and rc == ETIMEDOUT and 0.15 < dt < 1.0
    q.get(timeout=30)
    _join([a, b])
    # the lock and gate are free again
    c = CTX.Process(target=workers.try_region, args=(shm_name, 1000, q))
    c.start()
    assert q.get(timeout=30)[1] == OK
    _join([c])


def test_drain_timeout_reopens_gate(shm_name):
    """A sibling op longer than the entry timeout: entry fails, and the gate
    is open again (a new submission is admitted at once)."""
    q = CTX.Queue()
    ready = CTX.Event()
    s = CTX.Process(target=workers.long_op_then_sleep, args=(shm_name, 3_000_000, ready))
    s.start()
    assert ready.wait(30)
    b = CTX.Process(target=workers.try_region, args=(shm_name, 300, q))
    b.start()
    tag, rc, dt, _ = q.get(timeout=30)
    assert rc == ETIMEDOUT and dt < 2.0
    _join([b])
    c = CTX.Process(target=workers.submit_once, args=(shm_name, 0, 0, q))
    c.start()
    _, rc, t0, t_admit, st = q.get(timeout=30)
    assert rc == OK and (t_admit - t0) < 50e6 and st["parks"] == 0
    _join([c])
    s.kill()
    s.join(10)


def test_dead_sibling_is_not_waited_for(shm_name):
    """A sibling killed with work in flight: the holder's liveness check
    clears its slot instead of waiting for the count."""
    q = CTX.Queue()
    ready = CTX.Event()
    s = CTX.Process(target=workers.long_op_then_sleep, args=(shm_name, 30_000_000, ready))
    s.start()
    assert ready.wait(30)
    os.kill(s.pid, signal.SIGKILL)
    s.join(10)
    b = CTX.Process(target=workers.try_region, args=(shm_name, 3000, q))
    b.start()
    tag, rc, dt, _ = q.get(timeout=30)
    assert rc == OK and dt < 1.0
    _join([b])


def test_dead_holder_is_recovered(shm_name):
    """The holder dies inside its region. A parked sibling notices, recovers
    the lock (robust mutex) and reopens the gate; later entries succeed."""
    q = CTX.Queue()
    ready = CTX.Event()
    h = CTX.Process(target=workers.hold_and_die, args=(shm_name, ready))
    h.start()
    assert ready.wait(30)
    s = CTX.Process(target=workers.submit_once, args=(shm_name, 0, 0, q))
    s.start()
    time.sleep(0.3)
    os.kill(h.pid, signal.SIGKILL)
    h.join(10)
    _, rc, t0, t_admit, st = q.get(timeout=30)
    assert rc == OK and st["parks"] == 1 and st["recoveries"] == 1
    _join([s])
    c = CTX.Process(target=workers.try_region, args=(shm_name, 2000, q))
    c.start()
    assert q.get(timeout=30)[1] == OK
    _join([c])


def test_dead_holder_recovered_by_next_entry(shm_name):
    q = CTX.Queue()
    ready = CTX.Event()
    h = CTX.Process(target=workers.hold_and_die, args=(shm_name, ready))
    h.start()
    assert ready.wait(30)
    os.kill(h.pid, signal.SIGKILL)
    h.join(10)
    c = CTX.Process(target=workers.try_region, args=(shm_name, 2000, q))
    c.start()
    tag, rc, dt, st = q.get(timeout=30)
    assert rc == RECOVERED and st["recoveries"] == 1
    _join([c])


def test_late_registration_waits_for_gate(shm_name):
    """A process that registers while the gate is closed is admitted only
    after the region ends."""
    q = CTX.Queue()
    ready = CTX.Event()
    a = CTX.Process(target=workers.hold_region, args=(shm_name, 0.6, ready, q))
    a.start()
    assert ready.wait(30)
    s = CTX.Process(target=workers.submit_once, args=(shm_name, 0, 0, q))
    s.start()
    res = _collect(q, 2)
    _join([a, s])
    t_end = [r for r in res if r[0] == "held"][0][1]
    sub = [r for r in res if r[0] == "submit"][0]
    assert sub[1] == OK and sub[3] >= t_end and sub[4]["parks"] == 1


def test_ungated_process_is_not_blocked(shm_name):
    q = CTX.Queue()
    ready = CTX.Event()
    a = CTX.Process(target=workers.hold_region, args=(shm_name, 0.6, ready, q))
    a.start()
    assert ready.wait(30)
    s = CTX.Process(target=workers.submit_once, args=(shm_name, 1, 0, q))
    s.start()
    res = _collect(q, 2)
    _join([a, s])
    t_end = [r for r in res if r[0] == "held"][0][1]
    sub = [r for r in res if r[0] == "submit"][0]
    assert sub[1] == OK and sub[3] < t_end and sub[4]["parks"] == 0 and sub[4]["gated"] == 0


def test_submission_timeout(shm_name):
    q = CTX.Queue()
    ready = CTX.Event()
    a = CTX.Process(target=workers.hold_region, args=(shm_name, 1.0, ready, q))
    a.start()
    assert ready.wait(30)
    s = CTX.Process(target=workers.submit_once, args=(shm_name, 0, 150_000_000, q))
    s.start()
    res = _collect(q, 2)
    _join([a, s])
    sub = [r for r in res if r[0] == "submit"][0]
    assert sub[1] == ETIMEDOUT


def test_state_errors(shm_name):
    L = harness.load()
    assert L.kg_region_begin(100) == ENOTATTACHED
    assert L.kg_region_end() == ENOTATTACHED
    assert L.kg_attach(shm_name.encode(), 0) == OK
    assert L.kg_attach(shm_name.encode(), 0) == ESTATE
    assert L.kg_region_end() == ESTATE
    assert L.kg_region_begin(100) == OK
    assert L.kg_region_begin(100) == ESTATE
    assert L.kg_detach() == ESTATE              # inside a region
    assert L.kg_region_end() == OK
    assert L.kg_detach() == OK
    assert L.kg_detach() == ESTATE


def test_foreign_segment_rejected(shm_name):
    with open("/dev/shm" + shm_name, "wb") as f:
        f.write(b"\0" * 100)
    L = harness.load()
    assert L.kg_attach(shm_name.encode(), 0) == EPEER


def _stop_all(procs):
    for p in procs:
        if p.is_alive():
            try:
                os.kill(p.pid, signal.SIGCONT)
            except ProcessLookupError:
                pass


def test_cpu_exclusive_region_stops_sibling_trees(shm_name):
    """Section 4.2, steps 4, 5 and 7: inside a CPU-exclusive region the other
    registered processes and their children make no CPU progress, the
    entering thread runs on one core, and both are undone at exit."""
    q = CTX.Queue()
    stop = CTX.Event()
    c_par = [CTX.RawValue("Q", 0) for _ in range(2)]
    c_kid = [CTX.RawValue("Q", 0) for _ in range(2)]
    readies = [CTX.Event() for _ in range(2)]
    sibs = [CTX.Process(target=workers.spinner, args=(shm_name, c_par[i], c_kid[i], readies[i], stop))
            for i in range(2)]
    holder = None
    try:
        for p in sibs:
            p.start()
        for r in readies:
            assert r.wait(60)
        holder = CTX.Process(target=workers.exclusive_holder,
                             args=(shm_name, c_par + c_kid, 4, 150, q))
        holder.start()
        tag, before, res = q.get(timeout=60)
        holder.join(60)
        assert holder.exitcode == 0
    finally:
        _stop_all(sibs + ([holder] if holder else []))
        stop.set()
    _join(sibs)
    assert tag == "excl" and len(res) == 4
    for c0, c1, c2, aff_in, aff_out, frozen in res:
        assert c1 == c0, "a stopped process advanced inside the region: %s -> %s" % (c0, c1)
        assert all(b > a for a, b in zip(c1, c2)), "not resumed after the region: %s -> %s" % (c1, c2)
        assert aff_in == 1 and aff_out == before
        assert frozen == 4                      # two registered processes, each with one child


def test_dead_cpu_exclusive_holder_resumes_siblings(shm_name):
    """Holder death (Section 4.2): the process that recovers the lock resumes
    the process trees the dead holder had stopped."""
    q = CTX.Queue()
    stop = CTX.Event()
    ready_s, ready_h = CTX.Event(), CTX.Event()
    c, ck = CTX.RawValue("Q", 0), CTX.RawValue("Q", 0)
    sib = CTX.Process(target=workers.spinner, args=(shm_name, c, ck, ready_s, stop))
    holder = None
    try:
        sib.start()
        assert ready_s.wait(60)
        holder = CTX.Process(target=workers.exclusive_hold_and_die, args=(shm_name, ready_h))
        holder.start()
        assert ready_h.wait(60)
        v0 = (c.value, ck.value)
        time.sleep(0.2)
        assert (c.value, ck.value) == v0            # stopped while the holder lives
        os.kill(holder.pid, signal.SIGKILL)
        holder.join(30)
        b = CTX.Process(target=workers.try_region, args=(shm_name, 5000, q))
        b.start()
        tag, rc, _, st = q.get(timeout=60)
        b.join(30)
        assert tag == "try" and rc == RECOVERED and st["recoveries"] == 1
        v1 = (c.value, ck.value)
        time.sleep(0.2)
        v2 = (c.value, ck.value)
        assert v2[0] > v1[0] and v2[1] > v1[1]      # resumed by the recovery
    finally:
        _stop_all([sib] + ([holder] if holder else []))
        stop.set()
    _join([sib])


def test_cpu_exclusive_holder_below_registered_parent(shm_name):
    """A holder whose parent is registered stops that parent's tree but not
    itself, so its regions complete."""
    q = CTX.Queue()
    dummy = CTX.RawValue("Q", 0)
    parent = CTX.Process(target=workers.registered_parent_of_holder, args=(shm_name, dummy, q))
    try:
        parent.start()
        tag, exitcode, got = q.get(timeout=120)
    finally:
        _stop_all([parent])
    _join([parent])
    assert tag == "parent" and exitcode == 0
    assert got[0] == "excl" and len(got[2]) == 2
    assert all(r[5] >= 1 for r in got[2])       # the parent (at least) was stopped


def test_failed_sibling_is_not_waited_for(shm_name):
    """Section 4.3: a context that failed its health check is retired; region
    entry does not wait for the work it still had in flight."""
    ready = CTX.Event()
    sib = CTX.Process(target=workers.long_op_then_fail, args=(shm_name, 3_000_000, ready))
    sib.start()
    try:
        assert ready.wait(30)
        q = CTX.Queue()
        b = CTX.Process(target=workers.try_region, args=(shm_name, 10000, q))
        b.start()
        tag, rc, dt, _ = q.get(timeout=60)
        b.join(30)
        assert tag == "try" and rc == OK and dt < 1.0, (rc, dt)
    finally:
        sib.kill()
        sib.join(30)


def test_failed_process_cannot_submit(shm_name):
    q = CTX.Queue()
    p = CTX.Process(target=workers.fail_then_submit, args=(shm_name, q))
    p.start()
    tag, rc = q.get(timeout=60)
    _join([p])
    assert tag == "failed_submit" and rc == -3       # KREX_EHIP


def test_region_revoked_after_its_lease(shm_name, monkeypatch):
    """Section 4.3 (time limits): with a 300 ms lease, a parked submitter
    reopens a region held for 1.5 s; the holder's exit reports the
    revocation; the holder's next, short region is not revoked (the
    revocation is bound to the region's gate word) and the sibling's next
    submission waits for it as usual."""
    monkeypatch.setenv("KREX_REGION_LEASE_MS", "300")
    q = CTX.Queue()
    ready, ready2 = CTX.Event(), CTX.Event()
    holder = CTX.Process(target=workers.hold_past_lease, args=(shm_name, 1.5, 200, ready, ready2, q))
    holder.start()
    assert ready.wait(30)
    sib = CTX.Process(target=workers.submit_twice, args=(shm_name, ready2, q))
    sib.start()
    res = _collect(q, 2)
    _join([holder, sib])
    h = [r for r in res if r[0] == "holder"][0]
    s = [r for r in res if r[0] == "sib"][0]
    _, rc1, rc2, t_in, t2_in, t2_out = h
    _, srw, t1, srw2, t2, st = s
    assert rc1 == -10 and rc2 == OK                 # KREX_EREVOKED, then a normal exit
    assert srw == OK and srw2 == OK
    assert 0.25e9 < t1 - t_in < 1.2e9               # admitted once the lease ran out
    assert st["revocations"] == 1
    assert t2 >= t2_out                             # the second region kept its exclusivity
