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
