"""The dispatch interceptor (libkrex_intercept.so through HSA_TOOLS_LIB)
gates a sibling that never calls this library: a torch process looping fp32
GEMMs. Every one of its gated batches runs between its admission and its
completion, and none of those intervals overlaps a critical region of the
holder (Section 5, the AMD variant: each admitted batch is counted until a
barrier packet behind it completes; Section 4.2, steps 2-3).
A process with the library loaded but no segment named passes everything
through."""
import json
import os
import subprocess
import sys
import time
import uuid

import pytest
import torch

import paper_2609_30057_amd as krex
from paper_2609_30057_amd.build import INTERCEPT_LIB

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SIBLING = r'''
import ctypes, json, os, sys, time
import torch
import paper_2609_30057_amd as krex
torch.cuda.init()
a = torch.randn(4096, 4096, device="cuda")
b = torch.randn_like(a)
torch.cuda.synchronize()
print("ready", flush=True)
end = time.monotonic() + float(sys.argv[1])
n = 0
while time.monotonic() < end:
    c = a @ b
    torch.cuda.synchronize()
    n += 1
class C(ctypes.Structure):
    _fields_ = [("batches", ctypes.c_uint64), ("dispatches", ctypes.c_uint64), ("passthrough", ctypes.c_uint64),
                ("timeouts", ctypes.c_uint64), ("errors", ctypes.c_uint64), ("active", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]
L = ctypes.CDLL(os.environ["HSA_TOOLS_LIB"])
st = C()
assert L.krex_intercept_stats(ctypes.byref(st)) == 0
cap = 1 << 16
ta = (ctypes.c_uint64 * cap)()
td = (ctypes.c_uint64 * cap)()
m = L.krex_intercept_log(ta, td, cap)
gs = krex.gate_stats() if st.active else {}
print(json.dumps({"iters": n, "stats": {k: getattr(st, k) for k, _ in C._fields_},
                  "log": [[ta[i], td[i]] for i in range(m)], "gate": gs}), flush=True)
'''


def _sibling(seconds, shm):
    env = dict(os.environ)
    env["HSA_TOOLS_LIB"] = INTERCEPT_LIB
    env["PYTHONPATH"] = ROOT + os.pathsep + env.get("PYTHONPATH", "")
    if shm:
        env["KREX_INTERCEPT_SHM"] = shm
    else:
        env.pop("KREX_INTERCEPT_SHM", None)
    return subprocess.Popen([sys.executable, "-c", SIBLING, str(seconds)], env=env, stdout=subprocess.PIPE,
                            stderr=subprocess.PIPE, text=True, cwd=ROOT)


def _finish(p):
    out, err = p.communicate(timeout=120)
    assert p.returncode == 0, err[-3000:]
    return json.loads(out.strip().splitlines()[-1])


@pytest.fixture
def shm_name():
    name = "/krex-itest-%s" % uuid.uuid4().hex[:12]
    yield name
    try:
        os.unlink("/dev/shm" + name)
    except FileNotFoundError:
        pass


def test_library_loaded_without_segment_passes_through():
    p = _sibling(0.5, None)
    assert p.stdout.readline().strip() == "ready"
    r = _finish(p)
    assert r["iters"] > 0 and r["stats"]["active"] == 0 and r["stats"]["batches"] == 0


def test_intercepted_sibling_never_runs_inside_regions(shm_name):
    krex.attach(shm_name=shm_name)
    p = None
    try:
        p = _sibling(4.0, shm_name)
        assert p.stdout.readline().strip() == "ready"
        time.sleep(0.3)
        windows, drains = [], []
        for _ in range(10):
            krex.region_begin()
            t_in = time.monotonic_ns()
            time.sleep(0.05)
            t_out = time.monotonic_ns()
            krex.region_end()
            windows.append((t_in, t_out))
            drains.append(krex.gate_stats()["last_drain_ns"])
            time.sleep(0.05)
        r = _finish(p)
        p = None
    finally:
        if p is not None:
            p.kill()
            p.wait(30)
        krex.detach()
    st = r["stats"]
    assert st["active"] == 1 and st["errors"] == 0 and st["timeouts"] == 0
    assert st["batches"] >= r["iters"] and st["dispatches"] >= st["batches"]
    log = r["log"]
    assert len(log) > 100
    for ta, td in log:
        assert ta <= td
        for a, b in windows:
            assert td <= a or ta >= b, "sibling batch [%d, %d] overlaps region [%d, %d]" % (ta, td, a, b)
    assert r["gate"]["parks"] > 0                  # the sibling met the closed gate
    assert max(drains) > 0                         # entries waited for its kernels
