"""MI355X (gfx950) hot path of a kernel benchmarking command.

Thin ctypes binding over ``libkrex.so`` (the C ABI in ``include/krex.h``):
argument marshalling only -- every step runs in the library's HIP kernels and
host code. PyTorch supplies device memory and streams.

Paper: KREX, "Concurrent Kernel Benchmarking on Shared GPUs via
Region-Granular Exclusivity". A benchmarking command generates inputs and
checks the candidate against a reference (values, shareable), then times it
in a loop that must own the GPU (Section 1; Section 2.1). The timed loop is
marked with ``region.critical()`` (Section 4.1) and entered with the
lock / gate / drain / flush protocol of Section 4.2.

Entry points: ``gen``, ``transform_words``, ``inject``, ``check``,
``flush``, ``probe``, ``attach`` / ``detach``, ``region.critical``,
``region_begin`` / ``region_end``, ``time_loop``, ``gate_stats``.
"""
import contextlib
import ctypes
import os
from dataclasses import dataclass

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkrex.so")

F32, BF16, F16, F8E4M3, U32 = 0, 1, 2, 3, 4
UNIFORM, NORMAL, BITCAST = 0, 1, 2
INJ_ROUND, INJ_EXACT = 0, 1
TL_REGION = 1
ATTACH_NO_GATE = 1
ATTACH_CPU_EXCLUSIVE = 2
PROBE_THREADS = 65536
PROBE_WAVES = 1024
PROBE_CLOCK_WORDS = 8

OK, RECOVERED = 0, 1
EINVAL, EALIGN, EHIP, ETIMEDOUT, ESTATE, ENOTATTACHED, ENOMEM, EPEER, ESYS, EREVOKED = (
    -1, -2, -3, -4, -5, -6, -7, -8, -9, -10)

_DISTS = {"uniform": UNIFORM, "normal": NORMAL, "bitcast": BITCAST}
_MODES = {"round": INJ_ROUND, "exact": INJ_EXACT}


class KrexError(RuntimeError):
    def __init__(self, status, what=""):
        self.status = status
        self.hip_error = None
        msg = "%s: %s (%d)" % (what, _strerror(status), status)
        if status == EHIP and _lib is not None:
            self.hip_error = int(_lib.krex_last_hip_error())
            msg += ", hipError %d" % self.hip_error
        super().__init__(msg)


class _CheckResult(ctypes.Structure):
    _fields_ = [("n", ctypes.c_uint64), ("mismatches", ctypes.c_uint64), ("nan_count", ctypes.c_uint64),
                ("argmax_abs", ctypes.c_uint64), ("max_abs", ctypes.c_float), ("max_rel", ctypes.c_float),
                ("reserved", ctypes.c_uint64 * 3)]


class _ProbeArgs(ctypes.Structure):
    _fields_ = [("iters", ctypes.c_uint64), ("sink", ctypes.c_void_p), ("clocks", ctypes.c_void_p)]


class _SgemmArgs(ctypes.Structure):
    _fields_ = [("M", ctypes.c_uint32), ("N", ctypes.c_uint32), ("K", ctypes.c_uint32),
                ("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("C", ctypes.c_void_p)]


class _GateStats(ctypes.Structure):
    _fields_ = [("regions", ctypes.c_uint64), ("last_drain_ns", ctypes.c_uint64),
                ("total_drain_ns", ctypes.c_uint64), ("parks", ctypes.c_uint64), ("park_ns", ctypes.c_uint64),
                ("recoveries", ctypes.c_uint64), ("last_frozen", ctypes.c_uint64), ("revocations", ctypes.c_uint64),
                ("slot", ctypes.c_int32), ("gated", ctypes.c_int32)]


LAUNCH_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_void_p)


@dataclass
class CheckResult:
    n: int
    mismatches: int
    nan_count: int
    argmax_abs: int
    max_abs: float
    max_rel: float

    def as_dict(self):
        return dict(n=self.n, mismatches=self.mismatches, nan_count=self.nan_count, argmax_abs=self.argmax_abs,
                    max_abs=self.max_abs, max_rel=self.max_rel)


CHECK_RESULT_BYTES = ctypes.sizeof(_CheckResult)
_lib = None


def lib():
    """The loaded libkrex.so. Raises if it has not been built: there is no
    fallback path."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libkrex.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        i32, u32, u64, f32, f64, vp = (ctypes.c_int32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float,
                                       ctypes.c_double, ctypes.c_void_p)
        sigs = {
            "krex_attach": (i32, [i32, ctypes.c_char_p, u32]),
            "krex_detach": (i32, []),
            "krex_gen": (i32, [vp, i32, u64, u64, u64, i32, f32, f32, vp]),
            "krex_gen_packed": (i32, [vp, i32, u64, u64, u64, i32, f32, f32, vp]),
            "krex_transform_words": (i32, [vp, i32, u64, vp, i32, f32, f32, vp]),
            "krex_inject": (i32, [vp, vp, i32, u64, u64, u64, f64, f32, i32, vp]),
            "krex_gen_inject": (i32, [vp, vp, i32, u64, u64, u64, i32, f32, f32, u64, u64, f64, f32, i32, vp]),
            "krex_check": (i32, [vp, i32, vp, i32, u64, f32, f32, vp, vp]),
            "krex_check_noalloc": (i32, [vp, i32, vp, i32, u64, f32, f32, vp, vp]),
            "krex_check_gen": (i32, [vp, i32, i32, u64, u64, u64, i32, f32, f32, f32, f32, vp, vp]),
            "krex_check_gen_packed": (i32, [vp, i32, i32, u64, u64, u64, i32, f32, f32, f32, f32, vp, vp]),
            "krex_flush": (i32, [vp, u64, u32, vp]),
            "krex_probe": (i32, [u64, vp, vp]),
            "krex_probe_clocked": (i32, [u64, vp, vp, vp]),
            "krex_region_begin": (i32, [vp, u32, vp, u64]),
            "krex_region_end": (i32, [vp]),
            "krex_time_loop": (i32, [LAUNCH_FN, vp, u32, u32, vp, u64, u32, u32, vp, vp, vp]),
            "krex_fixture_sgemm": (i32, [u32, u32, u32, vp, vp, vp, vp]),
            "krex_get_gate_stats": (i32, [vp]),
            "krex_health_check": (i32, [vp]),
            "krex_strerror": (ctypes.c_char_p, [i32]),
            "krex_last_hip_error": (i32, []),
            "krex_version": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sigs.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _strerror(st):
    if _lib is None:
        return "status"
    return _lib.krex_strerror(st).decode()


def _chk(st, what):
    if st < 0:
        raise KrexError(st, what)
    return st


def _torch():
    import torch
    return torch


def _stream(stream):
    if stream is None:
        return _torch().cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def dtype_code(dtype):
    torch = _torch()
    table = {torch.float32: F32, torch.bfloat16: BF16, torch.float16: F16, torch.float8_e4m3fn: F8E4M3,
             torch.int32: U32, torch.uint32: U32}
    if dtype not in table:
        raise ValueError("unsupported dtype %s" % dtype)
    return table[dtype]


def _dev(t):
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _dist(d):
    return _DISTS[d] if isinstance(d, str) else int(d)


# --------------------------------------------------------------------- generation

def gen(t, seed, offset=0, dist="uniform", p0=None, p1=None, stream=None):
    """Fills tensor t with element j = transform(W_seed[offset + j]) (Philox4x32-10).
    uniform: [p0, p1) (default [-1, 1)); normal: mean p0, std p1 (default 0, 1);
    bitcast: raw 32-bit patterns as fp32 values."""
    d = _dist(dist)
    if p0 is None:
        p0 = -1.0 if d == UNIFORM else 0.0
    if p1 is None:
        p1 = 1.0 if d == UNIFORM else (1.0 if d == NORMAL else 0.0)
    _chk(lib().krex_gen(_dev(t), dtype_code(t.dtype), t.numel(), seed & (2**64 - 1), offset, d, p0, p1,
                        _stream(stream)), "krex_gen")
    return t


def gen_packed(t, seed, offset=0, dist="uniform", p0=None, p1=None, stream=None):
    """Packed-stream generation for bf16 / fp16 / fp8 tensors: element j uses
    the 16- or 8-bit field offset + j of the Philox word stream (bitcast:
    the field's bits)."""
    d = _dist(dist)
    if p0 is None:
        p0 = -1.0 if d == UNIFORM else 0.0
    if p1 is None:
        p1 = 1.0 if d == UNIFORM else (1.0 if d == NORMAL else 0.0)
    _chk(lib().krex_gen_packed(_dev(t), dtype_code(t.dtype), t.numel(), seed & (2**64 - 1), offset, d, p0, p1,
                               _stream(stream)), "krex_gen_packed")
    return t


def transform_words(t, words, dist="uniform", p0=None, p1=None, stream=None):
    d = _dist(dist)
    if p0 is None:
        p0 = -1.0 if d == UNIFORM else 0.0
    if p1 is None:
        p1 = 1.0 if d == UNIFORM else (1.0 if d == NORMAL else 0.0)
    if words.numel() != t.numel():
        raise ValueError("words and t must have the same number of elements")
    _chk(lib().krex_transform_words(_dev(t), dtype_code(t.dtype), t.numel(), _dev(words), d, p0, p1,
                                    _stream(stream)), "krex_transform_words")
    return t


def inject(y, x, mask_seed, rate, delta, mode="exact", mask_offset=0, stream=None):
    """y = x with a Bernoulli(rate) mask of elements perturbed by delta (ROUND or EXACT mode)."""
    if y.dtype != x.dtype or y.numel() != x.numel():
        raise ValueError("x and y must have the same dtype and size")
    m = _MODES[mode] if isinstance(mode, str) else int(mode)
    _chk(lib().krex_inject(_dev(y), _dev(x), dtype_code(x.dtype), x.numel(), mask_seed & (2**64 - 1),
                           mask_offset, float(rate), float(delta), m, _stream(stream)), "krex_inject")
    return y


def gen_inject(x, y, seed, offset=0, dist="uniform", p0=None, p1=None, mask_seed=0, rate=0.0, delta=0.0,
               mode="exact", mask_offset=0, stream=None):
    """x = gen(x, seed, offset, dist, p0, p1) and y = inject(y, x, mask_seed,
    rate, delta, mode, mask_offset) in one call (one pass when both offsets
    are multiples of 4)."""
    if y.dtype != x.dtype or y.numel() != x.numel():
        raise ValueError("x and y must have the same dtype and size")
    d = _dist(dist)
    if p0 is None:
        p0 = -1.0 if d == UNIFORM else 0.0
    if p1 is None:
        p1 = 1.0 if d == UNIFORM else (1.0 if d == NORMAL else 0.0)
    m = _MODES[mode] if isinstance(mode, str) else int(mode)
    _chk(lib().krex_gen_inject(_dev(x), _dev(y), dtype_code(x.dtype), x.numel(), seed & (2**64 - 1), offset, d, p0,
                               p1, mask_seed & (2**64 - 1), mask_offset, float(rate), float(delta), m,
                               _stream(stream)), "krex_gen_inject")
    return x, y


def check_result_buffer(device=None):
    """A device buffer for one check result (64 bytes)."""
    torch = _torch()
    return torch.empty(CHECK_RESULT_BYTES, dtype=torch.uint8, device=device or "cuda")


def decode_check_result(buf):
    raw = bytes(buf.cpu().numpy().tobytes())
    r = _CheckResult.from_buffer_copy(raw)
    return CheckResult(int(r.n), int(r.mismatches), int(r.nan_count), int(r.argmax_abs), float(r.max_abs),
                       float(r.max_rel))


def check(a, b, rtol, atol, out=None, stream=None, sync=True):
    """allclose check of candidate a against reference b (b's magnitude scales rtol).
    With sync=False returns the device result buffer to decode later."""
    if a.numel() != b.numel():
        raise ValueError("a and b must have the same number of elements")
    if out is None:
        out = check_result_buffer(a.device)
    _chk(lib().krex_check(_dev(a), dtype_code(a.dtype), _dev(b), dtype_code(b.dtype), a.numel(), float(rtol),
                          float(atol), _dev(out), _stream(stream)), "krex_check")
    if not sync:
        return out
    return decode_check_result(out)


def check_noalloc(a, b, rtol, atol, out, stream=None, sync=True):
    """check() through krex_check_noalloc: the library allocates nothing (its
    partials live in a fixed device array shared by every call on the GPU;
    overlapping calls on one GPU race). `out` is the caller's result buffer
    (check_result_buffer()). With sync=False returns `out` undecoded."""
    if a.numel() != b.numel():
        raise ValueError("a and b must have the same number of elements")
    _chk(lib().krex_check_noalloc(_dev(a), dtype_code(a.dtype), _dev(b), dtype_code(b.dtype), a.numel(),
                                  float(rtol), float(atol), _dev(out), _stream(stream)), "krex_check_noalloc")
    if not sync:
        return out
    return decode_check_result(out)


def check_gen(a, dtype_b, seed, rtol, atol, offset=0, dist="uniform", p0=None, p1=None, out=None, stream=None,
              sync=True):
    """check(a, b, rtol, atol) for the b that gen(b, seed, offset, dist, p0,
    p1) would write into a tensor of dtype_b with a's size, regenerated
    instead of read (only a is read). With sync=False returns the device
    result buffer to decode later."""
    d = _dist(dist)
    if p0 is None:
        p0 = -1.0 if d == UNIFORM else 0.0
    if p1 is None:
        p1 = 1.0 if d == UNIFORM else (1.0 if d == NORMAL else 0.0)
    if out is None:
        out = check_result_buffer(a.device)
    _chk(lib().krex_check_gen(_dev(a), dtype_code(a.dtype), dtype_code(dtype_b), a.numel(), seed & (2**64 - 1), offset,
                              d, p0, p1, float(rtol), float(atol), _dev(out), _stream(stream)), "krex_check_gen")
    if not sync:
        return out
    return decode_check_result(out)


def check_gen_packed(a, dtype_b, seed, rtol, atol, offset=0, dist="uniform", p0=None, p1=None, out=None,
                     stream=None, sync=True):
    """check(a, b, rtol, atol) for the b that gen_packed(b, seed, offset,
    dist, p0, p1) would write into a bf16 / fp16 / fp8 tensor of a's size,
    regenerated instead of read (only a is read)."""
    d = _dist(dist)
    if p0 is None:
        p0 = -1.0 if d == UNIFORM else 0.0
    if p1 is None:
        p1 = 1.0 if d == UNIFORM else (1.0 if d == NORMAL else 0.0)
    if out is None:
        out = check_result_buffer(a.device)
    _chk(lib().krex_check_gen_packed(_dev(a), dtype_code(a.dtype), dtype_code(dtype_b), a.numel(),
                                     seed & (2**64 - 1), offset, d, p0, p1, float(rtol), float(atol), _dev(out),
                                     _stream(stream)), "krex_check_gen_packed")
    if not sync:
        return out
    return decode_check_result(out)


def flush(buf, pattern=0, stream=None):
    """Writes `pattern` to every 32-bit word of buf (16-byte multiple)."""
    _chk(lib().krex_flush(_dev(buf), buf.numel() * buf.element_size(), pattern & 0xFFFFFFFF, _stream(stream)),
         "krex_flush")


def _check_clock_buffer(clocks):
    t = _torch()
    if clocks.dtype != t.int64 or clocks.numel() < PROBE_WAVES * PROBE_CLOCK_WORDS or not clocks.is_contiguous():
        raise ValueError("clocks must be a contiguous int64 tensor of %d values" % (PROBE_WAVES * PROBE_CLOCK_WORDS))
    if clocks.data_ptr() % 16:
        raise ValueError("clocks must be 16-byte aligned")


def probe(iters, sink, stream=None, clocks=None):
    if sink.numel() < PROBE_THREADS or sink.dtype != _torch().float32:
        raise ValueError("sink must hold %d float32 values" % PROBE_THREADS)
    if clocks is None:
        _chk(lib().krex_probe(iters, _dev(sink), _stream(stream)), "krex_probe")
    else:
        _check_clock_buffer(clocks)
        _chk(lib().krex_probe_clocked(iters, _dev(sink), _dev(clocks), _stream(stream)), "krex_probe_clocked")


def probe_clocks(clocks):
    """Decodes one probe's clock record (a tensor filled by probe(...,
    clocks=) or a clocked probe_launcher) into numpy arrays per wave:
    cycles and real-time ticks (100 MHz) elapsed, the effective shader clock
    in MHz, the start and end real-time stamps, the XCD and the HW_ID."""
    import numpy as np
    a = clocks[:PROBE_WAVES * PROBE_CLOCK_WORDS].cpu().numpy().view(np.uint64).reshape(PROBE_WAVES, PROBE_CLOCK_WORDS)
    cyc = (a[:, 1] - a[:, 0]).astype(np.float64)
    rt = (a[:, 3] - a[:, 2]).astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        mhz = np.where(rt > 0, cyc / rt * 100.0, np.nan)
    return {"cycles": cyc, "rt_ticks": rt, "mhz": mhz, "rt_start": a[:, 2], "rt_end": a[:, 3],
            "xcc": (a[:, 6] & 0xF).astype(np.int64), "hw_id": a[:, 4].astype(np.int64)}


def fixture_sgemm(A, B, C, stream=None):
    M, K = A.shape
    K2, N = B.shape
    if K2 != K or tuple(C.shape) != (M, N):
        raise ValueError("shape mismatch")
    _chk(lib().krex_fixture_sgemm(M, N, K, _dev(A), _dev(B), _dev(C), _stream(stream)), "krex_fixture_sgemm")


# ----------------------------------------------------------------------- regions

def attach(device=None, shm_name=None, gated=True, cpu_exclusive=False):
    """Registers this process with its GPU's region coordinator (Section 4.2).
    ``cpu_exclusive`` makes this process's regions stop the other registered
    process trees and pin the entering thread (Section 4.2, steps 4-5, 7)."""
    if device is None:
        device = _torch().cuda.current_device()
    name = shm_name.encode() if shm_name else None
    flags = (0 if gated else ATTACH_NO_GATE) | (ATTACH_CPU_EXCLUSIVE if cpu_exclusive else 0)
    return _chk(lib().krex_attach(device, name, flags), "krex_attach")


def detach():
    return _chk(lib().krex_detach(), "krex_detach")


def region_begin(timeout_ms=60000, flush_buf=None, stream=None):
    fb = _dev(flush_buf) if flush_buf is not None else None
    fbytes = flush_buf.numel() * flush_buf.element_size() if flush_buf is not None else 0
    return _chk(lib().krex_region_begin(_stream(stream), timeout_ms, fb, fbytes), "krex_region_begin")


def region_end(stream=None):
    return _chk(lib().krex_region_end(_stream(stream)), "krex_region_end")


class region:
    """``with region.critical(): ...`` marks a critical region (Section 4.1)."""

    @staticmethod
    @contextlib.contextmanager
    def critical(timeout_ms=60000, flush_buf=None, stream=None):
        region_begin(timeout_ms, flush_buf, stream)
        try:
            yield
        finally:
            region_end(stream)


def health_check(stream=None):
    """Context health after a command (Section 4.3): raises KrexError and marks
    this process's slot failed if the context is no longer usable."""
    return _chk(lib().krex_health_check(_stream(stream)), "krex_health_check")


def gate_stats():
    s = _GateStats()
    _chk(lib().krex_get_gate_stats(ctypes.byref(s)), "krex_get_gate_stats")
    return {k: getattr(s, k) for k, _ in _GateStats._fields_}


# --------------------------------------------------------------------- timed loop

def probe_launcher(iters, sink, clocks=None):
    """(fn, user) for time_loop that launches the probe kernel from C;
    clocks: None or a device tensor of PROBE_WAVES * PROBE_CLOCK_WORDS int64
    (see probe_clocks)."""
    if clocks is not None:
        _check_clock_buffer(clocks)
    args = _ProbeArgs(iters, _dev(sink), _dev(clocks) if clocks is not None else None)
    fn = ctypes.cast(ctypes.cast(lib().krex_probe_launch, ctypes.c_void_p).value, LAUNCH_FN)
    return fn, args


def sgemm_launcher(A, B, C):
    M, K = A.shape
    N = B.shape[1]
    args = _SgemmArgs(M, N, K, _dev(A), _dev(B), _dev(C))
    fn = ctypes.cast(ctypes.cast(lib().krex_sgemm_launch, ctypes.c_void_p).value, LAUNCH_FN)
    return fn, args


def time_loop(fn, warmup, reps, flush_buf=None, region=False, timeout_ms=60000, stream=None, user=None,
              with_flush_times=False):
    """do_bench-style loop. fn is a Python callable taking no arguments (it
    launches on the given stream), or a (LAUNCH_FN, ctypes struct) pair from
    probe_launcher / sgemm_launcher. Returns the per-rep times in ms (and the
    per-rep flush times when with_flush_times)."""
    if isinstance(fn, tuple):
        cfn, user_struct = fn
        user_ptr = ctypes.cast(ctypes.byref(user_struct), ctypes.c_void_p)
    else:
        py = fn

        def _tramp(_user, _stream):
            py()

        cfn = LAUNCH_FN(_tramp)
        user_ptr = None
    times = (ctypes.c_float * reps)()
    ftimes = (ctypes.c_float * reps)()
    fb = _dev(flush_buf) if flush_buf is not None else None
    fbytes = flush_buf.numel() * flush_buf.element_size() if flush_buf is not None else 0
    _chk(lib().krex_time_loop(cfn, user_ptr, warmup, reps, fb, fbytes, TL_REGION if region else 0, timeout_ms,
                              _stream(stream), times, ftimes), "krex_time_loop")
    if with_flush_times:
        return list(times), list(ftimes)
    return list(times)


def version():
    return lib().krex_version().decode()
