"""Builds and loads the CPU harness of the region coordinator: gate.cpp (the
product source) plus fake_device.cpp, compiled with g++ into one shared
library. Variant "tsan" adds ThreadSanitizer (host code only)."""
import ctypes
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2609_30057_amd", "csrc")
SRCS = [os.path.join(CSRC, "gate.cpp"), os.path.join(HERE, "fake_device.cpp")]


def lib_path(variant=""):
    return os.path.join(HERE, "libgate_harness%s.so" % ("_" + variant if variant else ""))


def build(variant=""):
    out = lib_path(variant)
    if os.path.exists(out) and all(os.path.getmtime(out) >= os.path.getmtime(s) for s in SRCS):
        return out
    flags = ["-std=c++17", "-O1" if variant else "-O2", "-g", "-fPIC", "-shared", "-Wall",
             "-I" + os.path.join(ROOT, "include"), "-I" + CSRC]
    if variant == "tsan":
        flags.append("-fsanitize=thread")
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.run(["g++", *flags, *SRCS, "-o", tmp, "-lpthread", "-lrt"], check=True)
    os.replace(tmp, out)
    return out


class Stats(ctypes.Structure):
    _fields_ = [("regions", ctypes.c_uint64), ("last_drain_ns", ctypes.c_uint64),
                ("total_drain_ns", ctypes.c_uint64), ("parks", ctypes.c_uint64), ("park_ns", ctypes.c_uint64),
                ("recoveries", ctypes.c_uint64), ("last_frozen", ctypes.c_uint64), ("revocations", ctypes.c_uint64),
                ("slot", ctypes.c_int32), ("gated", ctypes.c_int32)]


def load(variant=""):
    L = ctypes.CDLL(build(variant))
    L.kg_attach.argtypes = [ctypes.c_char_p, ctypes.c_uint32]
    L.kg_submit.argtypes = [ctypes.c_uint32, ctypes.c_uint64, ctypes.POINTER(ctypes.c_uint64)]
    L.kg_wait_idle.argtypes = [ctypes.c_uint32]
    L.kg_region_begin.argtypes = [ctypes.c_uint32]
    L.kg_inflight.restype = ctypes.c_int64
    L.kg_now.restype = ctypes.c_uint64
    L.kg_stats.argtypes = [ctypes.POINTER(Stats)]
    L.kg_log_get.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(ctypes.c_uint64)]
    L.kg_fail.restype = None
    return L


def log(L):
    out = []
    s, e = ctypes.c_uint64(), ctypes.c_uint64()
    for i in range(L.kg_log_count()):
        L.kg_log_get(i, ctypes.byref(s), ctypes.byref(e))
        out.append((s.value, e.value))
    return out


def stats(L):
    st = Stats()
    L.kg_stats(ctypes.byref(st))
    return {k: getattr(st, k) for k, _ in Stats._fields_}
