"""Builds the host-only Philox cross-check helper (tests/pins/philox_xcheck.cpp)
with g++ from two published engine headers: rocRAND's and ATen's."""
import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "philox_xcheck.cpp")
LIB = os.path.join(HERE, "libphilox_xcheck.so")


def _torch_include():
    import torch.utils.cpp_extension as ce
    return ce.include_paths()[0]


def load():
    if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp%d" % os.getpid()
        subprocess.run(["g++", "-std=c++17", "-O2", "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__",
                        "-I/opt/rocm/include", "-I" + _torch_include(), SRC, "-o", tmp], check=True)
        os.replace(tmp, LIB)
    L = ctypes.CDLL(LIB)
    for f in (L.xc_rocrand_words, L.xc_aten_words):
        f.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p]
    return L


def rocrand_words(L, seed, offset, n):
    out = np.empty(n, dtype=np.uint32)
    L.xc_rocrand_words(seed, offset, n, out.ctypes.data)
    return out


def aten_words(L, seed, offset, n):
    out = np.empty(n, dtype=np.uint32)
    L.xc_aten_words(seed, offset, n, out.ctypes.data)
    return out
