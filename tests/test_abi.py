"""The C-ABI library loads on a host without a GPU and exports every function
include/krex.h declares (no compute calls here); the header's constants and
the result struct layout agree with the Python binding."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "krex.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(krex_[a-z_0-9]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def declared_constants():
    text = open(HEADER).read()
    return {m.group(1): int(m.group(2).replace("u", ""), 0)
            for m in re.finditer(r"#define\s+(KREX_[A-Z0-9_]+)\s+\(?(-?(?:0x)?[0-9A-Fa-f]+u?)\)?", text)}


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("krex_attach", "krex_detach", "krex_gen", "krex_inject", "krex_check", "krex_flush",
              "krex_region_begin", "krex_region_end", "krex_time_loop", "krex_probe", "krex_strerror"):
        assert n in names


def test_interceptor_exports_its_header():
    from paper_2609_30057_amd.build import INTERCEPT_LIB
    if not os.path.exists(INTERCEPT_LIB):
        pytest.fail("libkrex_intercept.so is not built; run __graft_entry__.build()")
    text = open(os.path.join(ROOT, "include", "krex_intercept.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = set(re.findall(r"^\s*[a-z_0-9]+\s*\*?\s*(krex_[a-z_0-9]+)\s*\(", text, flags=re.M))
    assert names == {"krex_intercept_stats", "krex_intercept_log"}
    L = ctypes.CDLL(INTERCEPT_LIB)
    for n in sorted(names) + ["OnLoad", "OnUnload"]:
        assert hasattr(L, n), n
    # loaded outside the HSA runtime it is inactive and reports so
    buf = (ctypes.c_uint64 * 6)()
    assert L.krex_intercept_stats(buf) == 0 and buf[5] == 0
    assert L.krex_intercept_log(None, None, 10) == 0


def test_library_exports_every_declared_function():
    from paper_2609_30057_amd import LIB_PATH
    if not os.path.exists(LIB_PATH):
        pytest.fail("libkrex.so is not built; run __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(L, n)]
    assert not missing, missing


def test_constants_match_binding():
    import paper_2609_30057_amd as k
    c = declared_constants()
    pairs = {"KREX_F32": k.F32, "KREX_BF16": k.BF16, "KREX_F16": k.F16, "KREX_F8E4M3": k.F8E4M3,
             "KREX_U32": k.U32, "KREX_UNIFORM": k.UNIFORM, "KREX_NORMAL": k.NORMAL, "KREX_BITCAST": k.BITCAST,
             "KREX_INJ_ROUND": k.INJ_ROUND, "KREX_INJ_EXACT": k.INJ_EXACT, "KREX_TL_REGION": k.TL_REGION,
             "KREX_ATTACH_NO_GATE": k.ATTACH_NO_GATE,
             "KREX_ATTACH_CPU_EXCLUSIVE": k.ATTACH_CPU_EXCLUSIVE,
             "KREX_EREVOKED": k.EREVOKED, "KREX_PROBE_THREADS": k.PROBE_THREADS,
             "KREX_PROBE_WAVES": k.PROBE_WAVES, "KREX_PROBE_CLOCK_WORDS": k.PROBE_CLOCK_WORDS,
             "KREX_OK": k.OK, "KREX_RECOVERED": k.RECOVERED, "KREX_EINVAL": k.EINVAL, "KREX_EALIGN": k.EALIGN,
             "KREX_EHIP": k.EHIP, "KREX_ETIMEDOUT": k.ETIMEDOUT, "KREX_ESTATE": k.ESTATE,
             "KREX_ENOTATTACHED": k.ENOTATTACHED, "KREX_ENOMEM": k.ENOMEM, "KREX_EPEER": k.EPEER,
             "KREX_ESYS": k.ESYS}
    for name, val in pairs.items():
        assert c[name] == val, name
    assert k.CHECK_RESULT_BYTES == 64


def test_host_only_entry_points():
    """Calls that touch no GPU: status strings, version, validation failures
    that return before any HIP call."""
    import paper_2609_30057_amd as k
    L = k.lib()
    assert L.krex_strerror(k.EINVAL) == b"invalid argument"
    assert b"gfx950" in L.krex_version()
    # bad dtype / misaligned pointer / bad tolerance are rejected before launching
    assert L.krex_gen(None, 9, 4, 0, 0, 0, -1.0, 1.0, None) == k.EINVAL
    assert L.krex_gen(ctypes.c_void_p(2), k.F32, 4, 0, 0, 0, -1.0, 1.0, None) == k.EALIGN
    assert L.krex_gen(None, k.F32, 4, 0, 2**64 - 2, 0, -1.0, 1.0, None) == k.EINVAL
    assert L.krex_gen(None, k.F32, 0, 0, 0, 0, 1.0, -1.0, None) == k.EINVAL
    # the packed stream exists for the narrow dtypes only
    assert L.krex_gen_packed(None, k.F32, 4, 0, 0, 0, -1.0, 1.0, None) == k.EINVAL
    assert L.krex_gen_packed(None, k.U32, 4, 0, 0, 0, -1.0, 1.0, None) == k.EINVAL
    assert L.krex_gen_packed(ctypes.c_void_p(1), k.F16, 4, 0, 0, 0, -1.0, 1.0, None) == k.EALIGN
    assert L.krex_gen_packed(None, k.F8E4M3, 4, 0, 0, 1, 0.0, -1.0, None) == k.EINVAL
    assert L.krex_gen_packed(None, k.BF16, 0, 0, 0, 0, -1.0, 1.0, None) == k.OK
    assert L.krex_check(None, k.F32, None, k.F32, 4, -1.0, 0.0, ctypes.c_void_p(8), None) == k.EINVAL
    assert L.krex_check(None, k.F32, None, k.F32, 2**33, 0.0, 0.0, ctypes.c_void_p(8), None) == k.EINVAL
    # the regenerated-reference check validates like generation and the check
    assert L.krex_check_gen(None, k.F32, k.U32, 4, 0, 0, 0, -1.0, 1.0, 0.0, 0.0, ctypes.c_void_p(8), None) == k.EINVAL
    assert L.krex_check_gen(None, k.F32, k.F16, 4, 0, 0, 0, 1.0, -1.0, 0.0, 0.0, ctypes.c_void_p(8), None) == k.EINVAL
    assert L.krex_check_gen(None, k.F32, k.F16, 4, 0, 0, 1, 0.0, -1.0, 0.0, 0.0, ctypes.c_void_p(8), None) == k.EINVAL
    assert L.krex_check_gen(None, k.F32, k.F16, 4, 0, 0, 0, -1.0, 1.0, float("nan"), 0.0, ctypes.c_void_p(8),
                            None) == k.EINVAL
    assert L.krex_check_gen(None, k.F32, k.F16, 2**33, 0, 0, 0, -1.0, 1.0, 0.0, 0.0, ctypes.c_void_p(8),
                            None) == k.EINVAL
    assert L.krex_check_gen(None, k.F32, k.F16, 4, 0, 2**64 - 2, 0, -1.0, 1.0, 0.0, 0.0, ctypes.c_void_p(8),
                            None) == k.EINVAL
    assert L.krex_check_gen(None, k.F32, k.F16, 4, 0, 0, 0, -1.0, 1.0, 0.0, 0.0, None, None) == k.EINVAL
    assert L.krex_check_gen(None, k.F32, k.F16, 4, 0, 0, 0, -1.0, 1.0, 0.0, 0.0, ctypes.c_void_p(8), None) == k.EINVAL
    assert L.krex_check_gen(ctypes.c_void_p(2), k.F32, k.F16, 4, 0, 0, 0, -1.0, 1.0, 0.0, 0.0, ctypes.c_void_p(8),
                            None) == k.EALIGN
    assert L.krex_check_gen(ctypes.c_void_p(16), k.F32, k.F16, 4, 0, 0, 0, -1.0, 1.0, 0.0, 0.0, ctypes.c_void_p(12),
                            None) == k.EALIGN
    # the packed-stream reference exists for the narrow dtypes only
    assert L.krex_check_gen_packed(None, k.F32, k.F32, 4, 0, 0, 0, -1.0, 1.0, 0.0, 0.0, ctypes.c_void_p(8),
                                   None) == k.EINVAL
    assert L.krex_check_gen_packed(None, k.F32, k.F8E4M3, 4, 0, 0, 1, 0.0, -1.0, 0.0, 0.0, ctypes.c_void_p(8),
                                   None) == k.EINVAL
    assert L.krex_check_gen_packed(ctypes.c_void_p(2), k.F32, k.BF16, 4, 0, 0, 0, -1.0, 1.0, 0.0, 0.0,
                                   ctypes.c_void_p(8), None) == k.EALIGN
    assert L.krex_inject(None, None, k.F16, 4, 0, 0, 1.5, 0.5, 1, None) == k.EINVAL
    assert L.krex_flush(None, 17, 0, None) == k.EINVAL
    assert L.krex_probe_clocked(10, ctypes.c_void_p(16), None, None) == k.EINVAL
    assert L.krex_probe_clocked(10, ctypes.c_void_p(16), ctypes.c_void_p(8), None) == k.EALIGN
    assert L.krex_check_noalloc(None, k.F32, None, k.F32, 2**33, 0.0, 0.0, ctypes.c_void_p(8), None) == k.EINVAL
    assert L.krex_check_noalloc(ctypes.c_void_p(16), k.F32, ctypes.c_void_p(16), k.F32, 4, 0.0, 0.0,
                                ctypes.c_void_p(12), None) == k.EALIGN
    assert L.krex_region_begin(None, 10, None, 0) == k.ENOTATTACHED
    assert L.krex_region_end(None) == k.ENOTATTACHED
    assert L.krex_detach() == k.ESTATE
