"""Chunked submission (KREX_CHUNK_BYTES): a gated process splits large
generation, injection and flush calls into separately admitted launches with
at most KREX_CHUNK_DEPTH in flight. The values must not change: a child
process (the settings are read once per process) runs every chunked entry
point on sizes spanning many 1 MiB chunks plus a ragged tail, at aligned and
unaligned offsets, and compares each output with the oracle bit for bit."""
import os
import subprocess
import sys
import uuid

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r'''
import sys
sys.path.insert(0, sys.argv[1])
import numpy as np
import torch
import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import assert_bits_equal, empty, to_storage

torch.cuda.set_device(0)
krex.attach(0, shm_name=sys.argv[2])
n = (3 << 20) + 77
print("chunked: gen f16 uniform n=%d offset 5" % n, flush=True)
x = empty("f16", n)
krex.gen(x, 2, 5, "uniform", -4.0, 4.0)
xr = oracle.gen("f16", n, 2, 5, 0, -4.0, 4.0)
assert_bits_equal(to_storage(x, "f16"), xr, "gen f16")
print("chunked: gen f32 normal offset 3", flush=True)
z = empty("f32", n)
krex.gen(z, 9, 3, "normal", 0.0, 1.0)
assert_bits_equal(to_storage(z, "f32"), oracle.gen("f32", n, 9, 3, 1, 0.0, 1.0), "gen f32 normal")
print("chunked: inject f16 exact", flush=True)
y = torch.empty_like(x)
krex.inject(y, x, 3, 0.01, 0.5, "exact", mask_offset=8)
yr, _ = oracle.inject(xr, "f16", 3, 0.01, 0.5, oracle.INJ_EXACT, 8)
assert_bits_equal(to_storage(y, "f16"), yr, "inject f16")
print("chunked: gen_inject f8 round", flush=True)
x8 = empty("f8", n)
y8 = empty("f8", n)
krex.gen_inject(x8, y8, 4, 0, "normal", 0.0, 1.0, mask_seed=6, rate=0.02, delta=0.25, mode="round")
x8r = oracle.gen("f8", n, 4, 0, 1, 0.0, 1.0)
y8r, _ = oracle.inject(x8r, "f8", 6, 0.02, 0.25, oracle.INJ_ROUND, 0)
assert_bits_equal(to_storage(x8, "f8"), x8r, "gen_inject x")
assert_bits_equal(to_storage(y8, "f8"), y8r, "gen_inject y")
print("chunked: gen_packed bf16 uniform", flush=True)
xb = empty("bf16", n)
krex.gen_packed(xb, 7, 16, "uniform", -1.0, 1.0)
assert_bits_equal(to_storage(xb, "bf16"), oracle.gen_packed("bf16", n, 7, 16, 0, -1.0, 1.0), "gen_packed")
print("chunked: flush 8 MiB + 48 B", flush=True)
fl = torch.empty(((8 << 20) + 48) // 4, dtype=torch.int32, device="cuda")
krex.flush(fl, 0x12345678)
torch.cuda.synchronize()
got = fl.cpu().numpy().view(np.uint32)
assert np.all(got == 0x12345678), "flush content"
print("chunked ok", flush=True)
krex.detach()
'''


def test_chunked_submissions_write_the_same_values():
    shm = "/krex-chunk-%s" % uuid.uuid4().hex[:10]
    env = dict(os.environ, KREX_CHUNK_BYTES=str(1 << 20), KREX_CHUNK_DEPTH="2")
    r = subprocess.run([sys.executable, "-c", CHILD, ROOT, shm], env=env, capture_output=True, text=True,
                       timeout=300)
    try:
        os.unlink("/dev/shm" + shm)
    except FileNotFoundError:
        pass
    assert r.returncode == 0 and "chunked ok" in r.stdout, (r.returncode, r.stdout[-2000:], r.stderr[-4000:])


CAPTURE_CHILD = r'''
import sys
sys.path.insert(0, sys.argv[1])
import torch
import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import assert_bits_equal, empty, to_storage

torch.cuda.set_device(0)
krex.attach(0, shm_name=sys.argv[2])
n = (3 << 20) + 77
x = empty("f16", n)
krex.gen(x, 2, 4, "uniform", -4.0, 4.0)          # eager first
torch.cuda.synchronize()
print("chunked capture: record", flush=True)
g = torch.cuda.CUDAGraph()
s = torch.cuda.Stream()
with torch.cuda.graph(g, stream=s, capture_error_mode="thread_local"):
    krex.gen(x, 2, 4, "uniform", -4.0, 4.0)
torch.cuda.synchronize()
xr = oracle.gen("f16", n, 2, 4, 0, -4.0, 4.0)
for rep in range(3):
    x.zero_()
    torch.cuda.synchronize()
    print("chunked capture: replay %d" % rep, flush=True)
    g.replay()
    torch.cuda.synchronize()
    assert_bits_equal(to_storage(x, "f16"), xr, "captured gen")
assert krex.health_check() == 0
del g
krex.detach()
print("capture ok", flush=True)
'''


def test_capture_is_not_chunked():
    """A gated process with chunking on records a large generation into a
    HIP graph: under capture the call is neither chunked nor counted (its
    launches only run when the graph does), and every replay writes the
    oracle's values."""
    shm = "/krex-chunkcap-%s" % uuid.uuid4().hex[:10]
    env = dict(os.environ, KREX_CHUNK_BYTES=str(1 << 20), KREX_CHUNK_DEPTH="2")
    r = subprocess.run([sys.executable, "-c", CAPTURE_CHILD, ROOT, shm], env=env, capture_output=True, text=True,
                       timeout=300)
    try:
        os.unlink("/dev/shm" + shm)
    except FileNotFoundError:
        pass
    assert r.returncode == 0 and "capture ok" in r.stdout, (r.returncode, r.stdout[-2000:], r.stderr[-4000:])
