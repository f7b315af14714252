"""Host-side pieces of bench.py that run without a GPU: the one-core pinning
of the oracle leg, the host facts beside it, and the refusal of more than
one GPU."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_pinned_core_pins_and_restores():
    before = os.sched_getaffinity(0)
    with bench.pinned_core() as pc:
        assert os.sched_getaffinity(0) == {pc.core}
        assert pc.core in before
    assert os.sched_getaffinity(0) == before


def test_host_facts():
    f = bench.host_facts()
    assert f["host_cpus"] == os.cpu_count()
    assert 1 <= f["allowed_cpus"] <= f["host_cpus"]
    assert "cpu_model" in f


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
