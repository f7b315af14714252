"""The region coordinator's multi-process CPU tests again, with every worker
process loading the ThreadSanitizer build of gate.cpp (libtsan preloaded into
the spawned interpreters only). The sanitizer sees each process's own
threads -- the caller and the fake device's completion thread, which
releases the in-flight counts -- and their accesses to the coordinator's
state; any report fails the worker (exit code 66) and leaves a log that
fails the test. Paper, Section 4.2: the counter is raised before the gate is
checked, and recovery of a dead holder is serialised with normal exit."""
import os
import subprocess
import uuid

import pytest

import tests.test_gate_cpu as base
from tests.gate import harness, workers


def _libtsan():
    try:
        path = subprocess.run(["g++", "-print-file-name=libtsan.so"], capture_output=True, text=True,
                              check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.fixture
def tsan(tmp_path, monkeypatch):
    lib = _libtsan()
    if lib is None:
        pytest.skip("libtsan is not available to g++ on this host")
    harness.build("tsan")
    log = tmp_path / "tsan"
    monkeypatch.setenv("LD_PRELOAD", lib)
    monkeypatch.setenv("TSAN_OPTIONS", "halt_on_error=1 exitcode=66 report_signal_unsafe=0 log_path=%s" % log)
    monkeypatch.setenv("KREX_GATE_VARIANT", "tsan")
    yield
    reports = sorted(tmp_path.glob("tsan*"))
    assert not reports, "ThreadSanitizer reports:\n" + "\n".join(r.read_text()[:6000] for r in reports)


@pytest.fixture
def shm_name():
    name = "/krex-tsan-%s" % uuid.uuid4().hex[:12]
    yield name
    try:
        os.unlink("/dev/shm" + name)
    except FileNotFoundError:
        pass


def test_workers_run_the_sanitized_build(tsan):
    """The spawned workers map libtsan and the ThreadSanitizer build of the
    coordinator (so the tests below are checked, not merely run)."""
    q = base.CTX.Queue()
    p = base.CTX.Process(target=workers.report_loaded, args=(q,))
    p.start()
    tag, has_tsan, has_build = q.get(timeout=60)
    base._join([p])
    assert tag == "loaded" and has_tsan and has_build


def test_no_sibling_work_runs_inside_regions_tsan(shm_name, tsan):
    base.test_no_sibling_work_runs_inside_regions(shm_name)


def test_dead_holder_is_recovered_tsan(shm_name, tsan):
    base.test_dead_holder_is_recovered(shm_name)


def test_region_revoked_after_its_lease_tsan(shm_name, tsan, monkeypatch):
    base.test_region_revoked_after_its_lease(shm_name, monkeypatch)
