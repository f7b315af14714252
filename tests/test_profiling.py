"""The profile summarisers on synthetic rocprofv3 output: the HBM traffic
table (copy-calibrated FETCH_SIZE / WRITE_SIZE, and exact read bytes from the
read-request counters by size) and the vector-issue model of the generation
kernels (per-unit instruction path of the gfx950 assembly, weighted by issue
cost, against the launch's waves and duration); and, in the same assembly,
the cache policy of every streaming 16-byte store."""
import csv
import json
import os

import pytest

from paper_2609_30057_amd import profiling as P

GIB = 1 << 30
FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
          "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
          "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _counters(path, rows):
    """rows: (kernel name, counter, value) per dispatch."""
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "pmc_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, FIELDS)
        w.writeheader()
        for i, (k, c, v) in enumerate(rows):
            w.writerow({"Correlation_Id": i, "Dispatch_Id": i, "Agent_Id": "Agent 1", "Queue_Id": 1, "Process_Id": 1,
                        "Thread_Id": 1, "Grid_Size": 256, "Kernel_Id": 1, "Kernel_Name": k, "Workgroup_Size": 256,
                        "LDS_Block_Size": 0, "Scratch_Size": 0, "VGPR_Count": 8, "Accum_VGPR_Count": 0,
                        "SGPR_Count": 16, "Counter_Name": c, "Counter_Value": v, "Start_Timestamp": 0,
                        "End_Timestamp": 1})


RATES = {"v_fma_f32": 2.0, "v_add_f32": 1.9, "v_add_u32": 1.9, "v_and_b32": 1.9, "v_lshrrev_b32": 1.8,
         "v_bitop3_b32": 1.9, "v_fmaak_f32": 1.9, "v_mul_f32": 1.9, "v_max_f32": 3.6, "v_max3_f32": 3.6,
         "v_cndmask_b32": 3.6, "v_perm_b32": 3.6, "v_bfe_u32": 3.6, "v_mul_hi_u32": 3.6, "v_mad_u64_u32": 3.7,
         "v_cvt_f32_u32": 3.6, "v_cvt_f32_f16": 3.6, "v_cvt_f32_fp8": 3.6, "v_cvt_pk_bf16_f32": 3.6,
         "v_cvt_pk_f16_f32": 3.6, "v_cmp_lt_f32": 3.7, "v_rcp_f32": 7.2, "v_sqrt_f32": 7.2,
         "v_cvt_pk_fp8_f32": 7.2}


class Args:
    def __init__(self, **kw):
        self.__dict__.update(kw)


def test_traffic_scales_by_the_copy_and_uses_exact_read_bytes(tmp_path):
    copy = "__amd_rocclr_copyBuffer"
    check = "void krex::k_check<1, 0, true, 2>(unsigned char const*)"
    flush = "krex::k_flush(HIP_vector_type<unsigned int, 4u>*, unsigned long, unsigned int)"
    # FETCH_SIZE counts a 128-byte request as 64 bytes: the 1 GiB copy reads as 512 MiB.
    _counters(tmp_path / "fetch", [(copy, "FETCH_SIZE", GIB / 2 / 1024), (check, "FETCH_SIZE", 60 * 1024),
                                   (flush, "FETCH_SIZE", 0.0)])
    _counters(tmp_path / "write", [(copy, "WRITE_SIZE", GIB / 1024), (check, "WRITE_SIZE", 0.0),
                                   (flush, "WRITE_SIZE", GIB / 1024)])
    # the check: 100 MiB in 128-byte requests plus 1 MiB in 64-byte ones
    _counters(tmp_path / "rdreq", [(copy, "TCC_EA0_RDREQ_32B_sum", 0), (copy, "TCC_EA0_RDREQ_64B_sum", 0),
                                   (copy, "TCC_EA0_RDREQ_128B_sum", GIB / 128),
                                   (check, "TCC_EA0_RDREQ_32B_sum", 0), (check, "TCC_EA0_RDREQ_64B_sum", 2**20 / 64),
                                   (check, "TCC_EA0_RDREQ_128B_sum", 100 * 2**20 / 128),
                                   (flush, "TCC_EA0_RDREQ_32B_sum", 0), (flush, "TCC_EA0_RDREQ_64B_sum", 0),
                                   (flush, "TCC_EA0_RDREQ_128B_sum", 0)])
    out, js = tmp_path / "t.md", tmp_path / "t.json"
    P.cmd_traffic(Args(fetch=str(tmp_path / "fetch"), write=str(tmp_path / "write"), rdreq=str(tmp_path / "rdreq"),
                       out=str(out), out_json=str(js), cmd="x", title="t", workload="w",
                       algo=json.dumps({"krex::k_check<1, 0, true, 2>": 100 * 2**20, "krex::k_flush": GIB})))
    data = json.load(open(js))
    assert data["calibration"]["fetch_scale"] == pytest.approx(2.0)
    assert data["calibration"]["write_scale"] == pytest.approx(1.0)
    chk = data["k_check/w"]
    assert chk["fetch_bytes"] == 101 * 2**20          # exact bytes, not 2 x 60 MiB
    assert chk["hbm_bytes_per_launch"] == 101 * 2**20
    assert data["k_flush/w"]["hbm_bytes_per_launch"] == GIB
    text = out.read_text()
    assert "1024.0 MiB read (1024 expected)" in text
    assert "| `krex::k_check<1, 0, true, 2>` | 1 | 120.0 | 101.0 | 0.0 | 100.0 | 1.010 |" in text


def test_issue_costs_cover_the_hot_instructions():
    rates = RATES
    assert P._op_cost("v_mad_u64_u32", rates) == 3.7
    assert P._op_cost("v_cndmask_b32_e64", rates) == 3.6        # encoding suffix dropped
    assert P._op_cost("v_fmac_f32_e32", rates) == 2.0            # fmac costs as fma
    assert P._op_cost("v_cmp_ge_u64_e32", rates) == 3.7          # compares cost as the measured compare
    assert P._op_cost("v_cvt_pk_fp8_f32", rates) == 7.2
    assert P._op_cost("v_xor_b32_e32", rates) == 1.9             # bitwise ops as v_and
    assert P._op_cost("v_sqrt_f32_e64", rates) == 7.2
    assert P._op_cost("v_unmeasured_op", rates) == 4.0


@pytest.fixture(scope="module")
def asm():
    """gfx950 assembly of kernels.hip, built with the library's flags."""
    from paper_2609_30057_amd import build as B
    return open(B.emit_asm(os.path.join(B.BUILD, "kernels_test.s"))).read()


def _kernel_body(asm, prefix):
    """(symbol, body) of every kernel whose mangled name starts with prefix."""
    import re
    return re.findall(r"^(" + re.escape(prefix) + r"\w*):(.*?)\.Lfunc_end", asm, re.S | re.M)


def test_store_cache_policies(asm):
    """Generated and injected outputs leave the Infinity Cache clean
    (non-temporal device-scope stores, nt sc1); only the flush allocates
    there (sc0 sc1), since evicting that cache is its job."""
    import re
    kinds = {"_ZN4krex5k_genI": "nt sc1", "_ZN4krex12k_gen_packedI": "nt sc1", "_ZN4krex8k_injectI": "nt sc1",
             "_ZN4krex12k_gen_injectI": "nt sc1", "_ZN4krex7k_flushE": "sc0 sc1"}
    for prefix, policy in kinds.items():
        bodies = _kernel_body(asm, prefix)
        assert bodies, prefix
        for sym, body in bodies:
            stores = re.findall(r"buffer_store_dwordx4[^\n]*", body)
            assert stores, sym
            assert all(st.rstrip().endswith(" " + policy) for st in stores), (sym, stores[:2])


def test_issue_model_of_a_generation_launch(tmp_path, asm):
    """The unit path of the fp32 uniform kernel (power-of-two range) holds
    Philox's 32x32->64 multiplies and three-way xors, and the model's time is
    waves x weighted cycles over 1024 SIMDs x 2.4 GHz."""
    ops = P._unit_path(asm, "_ZN4krex5k_genILi0ELi0ELb1EEEvNS_9GenParamsE")
    assert ops.count("v_mad_u64_u32") >= 18 and ops.count("v_bitop3_b32") >= 18
    assert any(o.startswith("v_fma") for o in ops)              # the fused uniform transform
    rates = {"cycles": RATES}
    rj = tmp_path / "rates.json"
    rj.write_text(json.dumps(rates))
    trace = tmp_path / "trace.csv"
    fields = ["Kind", "Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X"]
    with open(trace, "w", newline="") as f:
        w = csv.DictWriter(f, fields)
        w.writeheader()
        for _ in range(3):
            w.writerow({"Kind": "KERNEL_DISPATCH", "Kernel_Name": "void krex::k_gen<0, 0, true>(krex::GenParams)",
                        "Start_Timestamp": 1000, "End_Timestamp": 41000, "Grid_Size_X": 1 << 24})
    out = tmp_path / "m.md"
    P.cmd_valu_model(Args(rates=str(rj), trace=str(trace), out=str(out), cmd="x", title="t", cus=256))
    row = [l for l in out.read_text().splitlines() if "k_gen<0, 0, true>" in l][0].split("|")
    cyc = sum(P._op_cost(o, rates["cycles"]) for o in ops)
    waves = (1 << 24) / 64
    assert int(row[2]) == len(ops)
    assert float(row[5]) == pytest.approx(waves * cyc / (1024 * 2.4e9) * 1e6, abs=0.06)
    assert float(row[6]) == pytest.approx((1 << 24) * 16 / 8e12 * 1e6, abs=0.06)   # HBM time of 16 B per unit
    assert float(row[8]) == pytest.approx(40.0)


def test_throughput_table_from_kernel_stats(tmp_path):
    """Algorithmic bytes over the average duration, for the listed launches
    of bench.py --kernels; the check's final reduction is reported apart."""
    path = tmp_path / "stats.csv"
    rows = [("void krex::k_check<2, 2, true, 3>(unsigned char const*)", 23, 160000.0),
            ("krex::k_flush(HIP_vector_type<unsigned int, 4u>*, unsigned long, unsigned int)", 23, 134217.728),
            ("krex::k_check_final(krex::CheckPartial const*)", 46, 4000.0)]
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs", "StdDev"])
        for name, calls, avg in rows:
            w.writerow([name, calls, calls * avg, avg, 1.0, avg, avg, 0.0])
    out = tmp_path / "t.md"
    P.cmd_throughput(Args(csv=str(path), out=str(out), cmd="rocprofv3 x", note="", tail=""))
    text = out.read_text()
    # 1 GiB of fp16 x fp16 operands (2^28 elements, 4 bytes each) in 160 us
    assert "| check, fp16 x fp16, 268M | `krex::k_check<2, 2, true, 3>` | 160.0 | 6711 | 0.839 | HBM read |" in text
    assert "| flush, 1 GiB | `krex::k_flush` | 134.2 | 8000 | 1.000 | HBM write |" in text
    assert "| generation, fp32 uniform, 67M | `krex::k_gen<0, 0, true>` | - |" in text
    assert "46 calls, average 4.00 us" in text


def test_units_per_launch():
    """16-byte units: of the output for generation and injection, of the
    narrower operand for the checks."""
    algo = P.kernels_algo()
    assert P._units("krex::k_gen<2, 0, true>", algo["krex::k_gen<2, 0, true>"]) == 2**25
    assert P._units("krex::k_inject<2, 1>", algo["krex::k_inject<2, 1>"]) == 2**25
    assert P._units("krex::k_check<1, 0, true, 2>", algo["krex::k_check<1, 0, true, 2>"]) == 2**24 * 2 / 16
    assert P._units("krex::k_check<3, 3, true, 3>", algo["krex::k_check<3, 3, true, 3>"]) == 2**28 / 16
    assert P._units("krex::k_check_gen<1, 0, 1, false, true, 2>",
                    algo["krex::k_check_gen<1, 0, 1, false, true, 2>"]) == 2**24 * 2 / 16


def test_sq_table_from_counters(tmp_path):
    """Per-wave instruction counts, clock, resident and issue-waiting waves
    from one dispatch's SQ counters (8 XCDs, 256 CUs)."""
    d = tmp_path / "sq"
    d.mkdir()
    k = "void krex::k_check<3, 3, true, 3>(unsigned char const*)"
    us = 100.0
    cyc = 2.4e9 * us * 1e-6                       # 240,000 cycles per XCD
    vals = {"SQ_WAVES": 4096, "SQ_INSTS_VALU": 4096 * 500.0, "SQ_INSTS_SALU": 4096 * 50.0,
            "GRBM_GUI_ACTIVE": 8 * cyc, "SQ_WAVE_CYCLES": 3.0 * 1024 * cyc / 4, "SQ_WAIT_INST_ANY": 1024 * cyc / 4}
    with open(d / "sq_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, FIELDS)
        w.writeheader()
        for c, v in vals.items():
            w.writerow({"Correlation_Id": 1, "Dispatch_Id": 1, "Agent_Id": "Agent 1", "Queue_Id": 1,
                        "Process_Id": 1, "Thread_Id": 1, "Grid_Size": 4096 * 64, "Kernel_Id": 1, "Kernel_Name": k,
                        "Workgroup_Size": 256, "LDS_Block_Size": 0, "Scratch_Size": 0, "VGPR_Count": 8,
                        "Accum_VGPR_Count": 0, "SGPR_Count": 16, "Counter_Name": c, "Counter_Value": v,
                        "Start_Timestamp": 0, "End_Timestamp": int(us * 1000)})
    out = tmp_path / "sq.md"
    P.cmd_sq(Args(dir=str(d), out=str(out), cmd="rocprofv3 x", note="", tail="", cus=256, xcds=8))
    # 2^28 fp8 pairs = 2^24 units; 4096 waves x 500 x 64 / 2^24 = 7.8 per unit
    assert "| `k_check<3, 3, true, 3>` | 100.0 | 4096 | 500 | 50 | 8 | 2400 | 3.0 | 1.0 |" in out.read_text()


def test_issue_model_prices_philox_products_in_context(tmp_path, asm):
    """With the Philox block entries, a word-stream generator's products are
    priced at (lockstep block cost - 20 three-way xors) / 20 in the last two
    columns; without them those columns stay empty."""
    ops = P._unit_path(asm, "_ZN4krex5k_genILi0ELi0ELb1EEEvNS_9GenParamsE")
    cycles = dict(RATES)
    cycles[P.PHILOX_LOCKSTEP] = 20 * 1.9 + 20 * 7.0          # a product costs 7 cycles in context
    cycles[P.PHILOX_PAIR] = 20 * 1.9 + 20 * 8.0
    assert P.philox_mad_cost(cycles, "krex::k_gen<0, 0, true>") == pytest.approx(7.0)
    assert P.philox_mad_cost(cycles, "krex::k_gen_packed<2, 0, 2>") == pytest.approx(8.0)
    assert P.philox_mad_cost(cycles, "krex::k_gen_packed<3, 1, 0>") == pytest.approx(7.0)
    assert P.philox_mad_cost(RATES, "krex::k_gen<0, 0, true>") is None
    trace = tmp_path / "trace.csv"
    fields = ["Kind", "Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X"]
    with open(trace, "w", newline="") as f:
        w = csv.DictWriter(f, fields)
        w.writeheader()
        w.writerow({"Kind": "KERNEL_DISPATCH", "Kernel_Name": "void krex::k_gen<0, 0, true>(krex::GenParams)",
                    "Start_Timestamp": 1000, "End_Timestamp": 41000, "Grid_Size_X": 1 << 24})
    for rates, filled in ((cycles, True), (RATES, False)):
        rj = tmp_path / "rates.json"
        rj.write_text(json.dumps({"cycles": rates}))
        out = tmp_path / "m.md"
        P.cmd_valu_model(Args(rates=str(rj), trace=str(trace), out=str(out), cmd="x", title="t", cus=256))
        row = [l for l in out.read_text().splitlines() if "k_gen<0, 0, true>" in l][0].split("|")
        if filled:
            ctx = dict(rates, v_mad_u64_u32=7.0)
            cyc = sum(P._op_cost(o, ctx) for o in ops)
            assert float(row[10]) == pytest.approx((1 << 24) / 64 * cyc / (1024 * 2.4e9) * 1e6, abs=0.06)
        else:
            assert row[10].strip() == "-" and row[11].strip() == "-"
