"""krex_check_noalloc, the check for callers that cannot allocate, against
krex_check, field by field at 0 ULP (and the oracle on the same inputs):
two calls in a row on one stream, the second smaller than the first (it
reduces fewer partials than the first left in the shared fixed array), a
ragged misaligned call (element path), an empty call, and the size limit
rejected before any launch."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2609_30057_amd as krex
from tests.gpu_helpers import from_storage, same_result

pytestmark = pytest.mark.gpu


def _near_pair(dta, dtb, n, seed):
    bf = oracle.gen("f32", n, seed, 0, 1, 0.0, 1.0)
    af, _ = oracle.inject(bf, "f32", seed + 1, 0.02, 0.01, oracle.INJ_ROUND)
    a = oracle.from_f32(af, dta) if dta != "f32" else af
    b = oracle.from_f32(bf, dtb) if dtb != "f32" else bf
    return a, b


def _both(a, dta, b, dtb, rtol, atol, ga=None, gb=None):
    """(krex_check record, krex_check_noalloc record, oracle record)."""
    ga = from_storage(a, dta) if ga is None else ga
    gb = from_storage(b, dtb) if gb is None else gb
    out_ref = krex.check_result_buffer()
    out_na = krex.check_result_buffer()
    print("no-alloc check: %s x %s n=%d" % (dta, dtb, a.size), flush=True)
    r_ref = krex.check(ga, gb, rtol, atol, out=out_ref)
    r_na = krex.check_noalloc(ga, gb, rtol, atol, out=out_na)
    return r_ref, r_na, oracle.check(a, dta, b, dtb, rtol, atol)


def test_two_calls_second_smaller():
    # first call: many blocks, several tiles and a ragged tail
    a, b = _near_pair("f16", "f16", (3 << 20) + 13, 21)
    r_ref, r_na, ref = _both(a, "f16", b, "f16", 1e-3, 1e-3)
    same_result(r_na, r_ref.as_dict())
    same_result(r_na, ref)
    # second call, right after, on far fewer blocks and another dtype pair
    a2, b2 = _near_pair("bf16", "f32", 40001, 22)
    r_ref2, r_na2, ref2 = _both(a2, "bf16", b2, "f32", 1.6e-2, 1e-2)
    same_result(r_na2, r_ref2.as_dict())
    same_result(r_na2, ref2)
    assert r_na2.n == 40001


def test_misaligned_and_empty():
    n = 100003
    a, b = _near_pair("f32", "f8", n + 1, 23)
    ga = from_storage(a, "f32")[1:]          # 4-byte aligned, not 16: the element path
    gb = from_storage(b, "f8")[1:]
    r_ref, r_na, ref = _both(a[1:], "f32", b[1:], "f8", 1e-4, 1e-5, ga, gb)
    same_result(r_na, r_ref.as_dict())
    same_result(r_na, ref)
    e = torch.empty(0, dtype=torch.float16, device="cuda")
    out = krex.check_result_buffer()
    r = krex.check_noalloc(e, e, 1e-3, 1e-3, out=out)
    assert (r.n, r.mismatches, r.nan_count, r.argmax_abs, r.max_abs, r.max_rel) == (0, 0, 0, 2**64 - 1, 0.0, 0.0)


def test_size_limit_rejected_before_launch():
    x = torch.zeros(16, dtype=torch.float16, device="cuda")
    out = krex.check_result_buffer()
    out.fill_(0xAB)
    torch.cuda.synchronize()
    L = krex.lib()
    st = L.krex_check_noalloc(ctypes.c_void_p(x.data_ptr()), 2, ctypes.c_void_p(x.data_ptr()), 2, 1 << 33,
                              1e-3, 1e-3, ctypes.c_void_p(out.data_ptr()), None)
    assert st == -1      # KREX_EINVAL
    torch.cuda.synchronize()
    assert np.all(out.cpu().numpy() == 0xAB), "a rejected call launched nothing"


def _attach_unique():
    import uuid
    shm = "/krex-na-%s" % uuid.uuid4().hex[:10]
    krex.attach(0, shm_name=shm)
    return shm


def _release(shm):
    import os
    krex.detach()
    try:
        os.unlink("/dev/shm" + shm)
    except FileNotFoundError:
        pass


def test_gated_calls_beyond_the_event_pool():
    """Attached with gating, 150 calls enqueued back to back: more than the
    64 completion events krex_attach pools, so later calls find the pool in
    use and wait for their stream instead of creating events. Every record
    equals krex_check's."""
    a, b = _near_pair("f16", "f16", (1 << 20) + 5, 24)
    ga, gb = from_storage(a, "f16"), from_storage(b, "f16")
    shm = _attach_unique()
    try:
        print("no-alloc: 150 gated calls", flush=True)
        want = krex.check(ga, gb, 1e-3, 1e-3).as_dict()
        outs = [krex.check_result_buffer() for _ in range(150)]
        for o in outs:
            krex.check_noalloc(ga, gb, 1e-3, 1e-3, out=o, sync=False)
        torch.cuda.synchronize()
        for o in outs:
            same_result(krex.decode_check_result(o), want)
        assert krex.health_check() == 0
    finally:
        _release(shm)


@pytest.mark.parametrize("attached", [False, True], ids=["ungated", "gated"])
def test_graph_capture_replays(attached):
    """The call recorded into a HIP graph (the use the entry point exists
    for), replayed three times with eager work in between that changes the
    reference: every replay's record equals krex_check's on the same data.
    Attached with gating, the captured call is not counted, and the process
    stays healthy."""
    a, b = _near_pair("bf16", "f32", (1 << 20) + 3, 25)
    ga, gb = from_storage(a, "bf16"), from_storage(b, "f32")
    shm = _attach_unique() if attached else None
    try:
        out = krex.check_result_buffer()
        krex.check_noalloc(ga, gb, 1.6e-2, 1e-2, out=out)    # eager first: scratch address, grid caches
        torch.cuda.synchronize()
        print("no-alloc: capture (attached=%s)" % attached, flush=True)
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        with torch.cuda.graph(g, stream=s, capture_error_mode="thread_local"):
            krex.check_noalloc(ga, gb, 1.6e-2, 1e-2, out=out, sync=False)
        torch.cuda.synchronize()
        base = gb.clone()
        for rep in range(3):
            krex.inject(gb, base, 40 + rep, 0.01 * (rep + 1), 0.5, "round")   # eager: a new reference
            torch.cuda.synchronize()
            print("no-alloc: replay %d" % rep, flush=True)
            g.replay()
            torch.cuda.synchronize()
            got = krex.decode_check_result(out)
            same_result(got, krex.check(ga, gb, 1.6e-2, 1e-2).as_dict())
            assert got.mismatches > 0
        if attached:
            assert krex.health_check() == 0
            st = krex.gate_stats()
            assert st["gated"]
        del g
    finally:
        if attached:
            _release(shm)
