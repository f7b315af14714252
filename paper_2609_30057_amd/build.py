"""Builds the three shared libraries of the package with hipcc:

  libkrexgate.so       the region coordinator (gate.cpp, plain POSIX C++),
                       one instance per process for both libraries below;
  libkrex.so           the C ABI of include/krex.h: kernels.hip,
                       check_gen.hip and check_gen_packed.hip for gfx950
                       and api.cpp (host C++ against the HIP runtime);
  libkrex_intercept.so the ROCm tools library of include/krex_intercept.h
                       (loaded through HSA_TOOLS_LIB).

and the measurement program valu_rates (issue cost of the vector
instructions the kernels use, run by bench.py --valu-rates).

The .hip sources are compiled as HIP for --offload-arch=gfx950; the rest is host
C++. Floating-point flags fix the semantics
the generated values and check verdicts are defined with: no contraction
into fused multiply-adds except where written, correctly rounded fp32
division and square root, fp32 denormals kept. Packed fp32 instructions are
disabled for all device code.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libkrex.so")
GATE_LIB = os.path.join(HERE, "libkrexgate.so")
INTERCEPT_LIB = os.path.join(HERE, "libkrex_intercept.so")
VALU_RATES = os.path.join(HERE, "valu_rates")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = ["-O3", "-std=c++17", "-fPIC", "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
          "-Wall", "-Wno-unused-function"]
DEVICE = ["-x", "hip", "--offload-arch=" + ARCH, "-ffp-contract=off",
          "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST = ["-x", "c++", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]

# The HSA tools header includes its siblings by bare name under this macro.
INTERCEPT = HOST + ["-DAMD_INTERNAL_BUILD", "-I/opt/rocm/include/hsa"]

SOURCES = [("kernels.hip", DEVICE), ("check_gen.hip", DEVICE), ("check_gen_packed.hip", DEVICE), ("api.cpp", HOST),
           ("gate.cpp", HOST), ("intercept.cpp", INTERCEPT)]


def _compile(src, flags, verbose):
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *COMMON, *flags, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    return obj


def _link(out, objs, extra, verbose, linker=HIPCC):
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [linker, "-shared", "-fPIC", *objs, "-o", tmp, *extra]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        kernels, check_gen, check_gen_packed, api, gate, intercept = ex.map(
            lambda sf: _compile(sf[0], sf[1], verbose), SOURCES)
    rpath = ["-L" + HERE, "-lkrexgate", "-Wl,-rpath,$ORIGIN", "-lpthread", "-lrt"]
    # The coordinator and the interceptor are plain host code: linked without
    # the HIP runtime (the interceptor loads inside the HSA runtime's start).
    _link(GATE_LIB, [gate], ["-Wl,-soname,libkrexgate.so", "-lpthread", "-lrt"], verbose, linker="g++")
    _link(LIB, [kernels, check_gen, check_gen_packed, api], ["--offload-arch=" + ARCH, *rpath], verbose)
    _link(INTERCEPT_LIB, [intercept], rpath, verbose, linker="g++")
    tmp = VALU_RATES + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-O3", "-std=c++17", "-x", "hip", "--offload-arch=" + ARCH, "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", os.path.join(CSRC, "valu_rates.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    os.replace(tmp, VALU_RATES)
    return LIB


def emit_asm(out_path: str) -> str:
    """gfx950 assembly of kernels.hip with the library's device flags."""
    cmd = [HIPCC, *COMMON, *DEVICE, "--cuda-device-only", "-S", os.path.join(CSRC, "kernels.hip"), "-o", out_path]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    return out_path


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
