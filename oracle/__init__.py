"""CPU oracle for the benchmarking-command hot path -- TEST INFRASTRUCTURE.

Only the test suite, ``__graft_entry__.smoke()`` and ``bench.py``'s
cpu_baseline leg may import this package. The product package
(``paper_2609_30057_amd``) never imports it, and the two share no code.

This module is a thin numpy/ctypes wrapper over ``krex_oracle.c`` (plain
single-threaded C) plus the timing statistic of the paper's Eq. 1, written
with numpy in ``stats.py``. The C file's header states every definition and
the passage of the paper each one reads.

Parity pins (tests/test_oracle_*.py) tie each function to something other
than itself: two independent Philox engines from published library headers,
torch's CPU dtype conversions over large sweeps, fp64 libm over every
possible input of the own ln / sin / cos, closed forms, hand-derived golden
cases and invariants. The probe is pinned by exact rational arithmetic on
small cases.
"""
import ctypes
import os

import numpy as np

from . import build as _build

F32, BF16, F16, F8E4M3, U32 = 0, 1, 2, 3, 4
UNIFORM, NORMAL, BITCAST = 0, 1, 2
INJ_ROUND, INJ_EXACT = 0, 1

DTYPE_NAMES = {"f32": F32, "bf16": BF16, "f16": F16, "f8": F8E4M3, "u32": U32}
NP_STORAGE = {F32: np.float32, BF16: np.uint16, F16: np.uint16, F8E4M3: np.uint8, U32: np.uint32}
ITEMSIZE = {F32: 4, BF16: 2, F16: 2, F8E4M3: 1, U32: 4}


class CheckResult(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint64), ("mismatches", ctypes.c_uint64),
                ("nan_count", ctypes.c_uint64), ("argmax_abs", ctypes.c_uint64),
                ("max_abs", ctypes.c_float), ("max_rel", ctypes.c_float)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = _build.ensure_built()
        L = ctypes.CDLL(path)
        u32p = ctypes.POINTER(ctypes.c_uint32)
        vp = ctypes.c_void_p
        L.ko_philox4x32_10.argtypes = [u32p, u32p, u32p]
        L.ko_word.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.ko_word.restype = ctypes.c_uint32
        L.ko_words.argtypes = [vp, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64]
        L.ko_gen.argtypes = [vp, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                             ctypes.c_int, ctypes.c_float, ctypes.c_float]
        L.ko_gen.restype = ctypes.c_int
        L.ko_gen_packed.argtypes = [vp, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                    ctypes.c_int, ctypes.c_float, ctypes.c_float]
        L.ko_packed_width.argtypes = [ctypes.c_int, ctypes.c_int]
        L.ko_transform_words.argtypes = [vp, ctypes.c_int, ctypes.c_uint64, vp, ctypes.c_int,
                                         ctypes.c_float, ctypes.c_float]
        L.ko_transform_words.restype = ctypes.c_int
        L.ko_inject.argtypes = [vp, vp, ctypes.c_int, ctypes.c_uint64, ctypes.c_uint64,
                                ctypes.c_uint64, ctypes.c_double, ctypes.c_float, ctypes.c_int]
        L.ko_inject.restype = ctypes.c_int64
        L.ko_inject_threshold.argtypes = [ctypes.c_double]
        L.ko_inject_threshold.restype = ctypes.c_uint64
        L.ko_check.argtypes = [vp, ctypes.c_int, vp, ctypes.c_int, ctypes.c_uint64,
                               ctypes.c_float, ctypes.c_float, ctypes.POINTER(CheckResult)]
        L.ko_check.restype = ctypes.c_int
        L.ko_flush.argtypes = [vp, ctypes.c_uint64, ctypes.c_uint32]
        L.ko_flush.restype = ctypes.c_int
        L.ko_probe.argtypes = [ctypes.c_uint64, vp, ctypes.c_uint32]
        L.ko_sgemm.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32, vp, vp, vp]
        L.ko_convert_from_f32.argtypes = [vp, ctypes.c_int, vp, ctypes.c_uint64]
        L.ko_convert_to_f32.argtypes = [vp, vp, ctypes.c_int, ctypes.c_uint64]
        L.ko_ln.argtypes = [ctypes.c_float]
        L.ko_ln.restype = ctypes.c_float
        L.ko_sincos_2pi_q24.argtypes = [ctypes.c_uint32, ctypes.POINTER(ctypes.c_float),
                                        ctypes.POINTER(ctypes.c_float)]
        L.ko_normal_pair.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.POINTER(ctypes.c_float),
                                     ctypes.POINTER(ctypes.c_float)]
        L.ko_uniform.argtypes = [ctypes.c_uint32, ctypes.c_float, ctypes.c_float]
        L.ko_uniform.restype = ctypes.c_float
        L.ko_ln_many.argtypes = [vp, vp, ctypes.c_uint64]
        L.ko_sincos_many.argtypes = [vp, vp, vp, ctypes.c_uint64]
        L.ko_normal_pairs.argtypes = [vp, vp, ctypes.c_uint64]
        L.ko_uniform_many.argtypes = [vp, vp, ctypes.c_uint64, ctypes.c_float, ctypes.c_float]
        _lib = L
    return _lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def dtype_code(dt):
    return DTYPE_NAMES[dt] if isinstance(dt, str) else int(dt)


def philox(ctr, key):
    c = (ctypes.c_uint32 * 4)(*[int(v) & 0xFFFFFFFF for v in ctr])
    k = (ctypes.c_uint32 * 2)(*[int(v) & 0xFFFFFFFF for v in key])
    o = (ctypes.c_uint32 * 4)()
    lib().ko_philox4x32_10(c, k, o)
    return [int(v) for v in o]


def word(seed, w):
    return int(lib().ko_word(seed, w))


def words(n, seed, offset=0):
    out = np.empty(n, dtype=np.uint32)
    lib().ko_words(_ptr(out), n, seed, offset)
    return out


def gen(dt, n, seed, offset=0, dist=UNIFORM, p0=-1.0, p1=1.0):
    """Generated tensor as its storage array (float32, or uint16/uint8 bit patterns)."""
    dt = dtype_code(dt)
    out = np.empty(n, dtype=NP_STORAGE[dt])
    st = lib().ko_gen(_ptr(out), dt, n, seed, offset, dist, p0, p1)
    if st != 0:
        raise ValueError("ko_gen rejected its arguments (%d)" % st)
    return out


def packed_width(dt, dist):
    """Field width in bits of the packed stream for (dtype, distribution); 0 if none."""
    return int(lib().ko_packed_width(dtype_code(dt), dist))


def gen_packed(dt, n, seed, offset=0, dist=UNIFORM, p0=-1.0, p1=1.0):
    """Packed-stream tensor (narrow dtypes only) as its storage array; offset counts fields."""
    dt = dtype_code(dt)
    out = np.empty(n, dtype=NP_STORAGE[dt])
    st = lib().ko_gen_packed(_ptr(out), dt, n, seed, offset, dist, p0, p1)
    if st != 0:
        raise ValueError("ko_gen_packed rejected its arguments (%d)" % st)
    return out


def transform_words(dt, words_, dist=UNIFORM, p0=-1.0, p1=1.0):
    dt = dtype_code(dt)
    w = np.ascontiguousarray(words_, dtype=np.uint32)
    out = np.empty(w.size, dtype=NP_STORAGE[dt])
    st = lib().ko_transform_words(_ptr(out), dt, w.size, _ptr(w), dist, p0, p1)
    if st != 0:
        raise ValueError("ko_transform_words rejected its arguments (%d)" % st)
    return out


def inject(x, dt, mask_seed, rate, delta, mode=INJ_EXACT, mask_offset=0):
    """Returns (y, number of perturbed elements)."""
    dt = dtype_code(dt)
    x = np.ascontiguousarray(x)
    y = np.empty_like(x)
    k = lib().ko_inject(_ptr(y), _ptr(x), dt, x.size, mask_seed, mask_offset, rate, delta, mode)
    if k < 0:
        raise ValueError("ko_inject rejected its arguments (%d)" % k)
    return y, int(k)


def inject_threshold(rate):
    return int(lib().ko_inject_threshold(rate))


def check(a, dta, b, dtb, rtol, atol):
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    assert a.size == b.size
    r = CheckResult()
    st = lib().ko_check(_ptr(a), dtype_code(dta), _ptr(b), dtype_code(dtb), a.size,
                        rtol, atol, ctypes.byref(r))
    if st != 0:
        raise ValueError("ko_check rejected its arguments (%d)" % st)
    return r.as_dict()


def flush_fill(buf, pattern):
    st = lib().ko_flush(_ptr(buf), buf.nbytes, pattern)
    if st != 0:
        raise ValueError("ko_flush rejected its arguments")


def probe(iters, threads=65536):
    out = np.empty(threads, dtype=np.float32)
    lib().ko_probe(iters, _ptr(out), threads)
    return out


def sgemm(A, B):
    A = np.ascontiguousarray(A, dtype=np.float32)
    B = np.ascontiguousarray(B, dtype=np.float32)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    C = np.empty((M, N), dtype=np.float32)
    lib().ko_sgemm(M, N, K, _ptr(A), _ptr(B), _ptr(C))
    return C


def from_f32(x, dt):
    dt = dtype_code(dt)
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.size, dtype=NP_STORAGE[dt])
    lib().ko_convert_from_f32(_ptr(out), dt, _ptr(x), x.size)
    return out


def to_f32(h, dt):
    dt = dtype_code(dt)
    h = np.ascontiguousarray(h, dtype=NP_STORAGE[dt])
    out = np.empty(h.size, dtype=np.float32)
    lib().ko_convert_to_f32(_ptr(out), _ptr(h), dt, h.size)
    return out


def ln(x):
    return float(lib().ko_ln(x))


def sincos_2pi_q24(k):
    s, c = ctypes.c_float(), ctypes.c_float()
    lib().ko_sincos_2pi_q24(k, ctypes.byref(s), ctypes.byref(c))
    return s.value, c.value


def normal_pair(w0, w1):
    a, b = ctypes.c_float(), ctypes.c_float()
    lib().ko_normal_pair(w0, w1, ctypes.byref(a), ctypes.byref(b))
    return a.value, b.value


def uniform(word_, lo, hi):
    return float(lib().ko_uniform(word_, lo, hi))


def ln_many(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    lib().ko_ln_many(_ptr(x), _ptr(out), x.size)
    return out


def sincos_many(k):
    k = np.ascontiguousarray(k, dtype=np.uint32)
    s = np.empty(k.size, dtype=np.float32)
    c = np.empty(k.size, dtype=np.float32)
    lib().ko_sincos_many(_ptr(k), _ptr(s), _ptr(c), k.size)
    return s, c


def normal_pairs(w):
    w = np.ascontiguousarray(w, dtype=np.uint32)
    assert w.size % 2 == 0
    z = np.empty(w.size, dtype=np.float32)
    lib().ko_normal_pairs(_ptr(w), _ptr(z), w.size // 2)
    return z


def uniform_many(w, lo, hi):
    w = np.ascontiguousarray(w, dtype=np.uint32)
    out = np.empty(w.size, dtype=np.float32)
    lib().ko_uniform_many(_ptr(w), _ptr(out), w.size, lo, hi)
    return out
