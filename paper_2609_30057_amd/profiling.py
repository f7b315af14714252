"""Summaries of rocprofv3 output (CSV) for the committed profiles.

  python -m paper_2609_30057_amd.profiling stats  --csv DIR/..._kernel_stats.csv --out FILE.md --cmd "..."
  python -m paper_2609_30057_amd.profiling traffic --fetch DIR --write DIR --out-json profiles/traffic.json
                                                 --out FILE.md --cmd "..."
  python -m paper_2609_30057_amd.profiling select --trace DIR/..._kernel_trace.csv --out FILE.md --cmd "..."
                                                 NAME[@GRID] ...
  python -m paper_2609_30057_amd.profiling valu-model --rates RATES.json --trace DIR/..._kernel_trace.csv
                                                 --out FILE.md --cmd "..."
  python -m paper_2609_30057_amd.profiling throughput --csv DIR/..._kernel_stats.csv --out FILE.md --cmd "..."
  python -m paper_2609_30057_amd.profiling sq --dir DIR --out FILE.md --cmd "..."

valu-model: for the one-unit-per-thread kernels (generation), the vector
instructions of the per-unit path in the gfx950 assembly (from the loop head
to the 16-byte store), each weighted by its measured issue cost (cycles per
wave64 instruction, bench.py --valu-rates), times the waves of the launch in
the kernel trace, over 4 SIMDs per CU x CUs x 2.4 GHz: the time the launch
needs at full vector issue, compared with its measured duration.

traffic: per-dispatch FETCH_SIZE and WRITE_SIZE (KiB) of each kernel, scaled by
what the same counters read for a plain device copy of 1 GiB (1 GiB fetched,
1 GiB written), and compared with the kernel's algorithmic bytes. With
--rdreq, a third pass of the read-request counters by size
(TCC_EA0_RDREQ_32B/64B/128B) gives the bytes read exactly: on gfx950
FETCH_SIZE counts a 128-byte request as 64 bytes, so the copy's factor of 2
is only right for kernels whose reads are all 128-byte requests.
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import re
import statistics

GIB = 1 << 30
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNELS_HIP = os.path.join(ROOT, "paper_2609_30057_amd", "csrc", "kernels.hip")
DEVICE_HPP = os.path.join(ROOT, "paper_2609_30057_amd", "csrc", "krex_device.hpp")
CHECK_HPP = os.path.join(ROOT, "paper_2609_30057_amd", "csrc", "check_device.hpp")

# kernels.hip is split into sections by "// ---- <name>" rules; a traffic
# figure is tied to the source of its kernel's section (plus the device
# header for the kernels that use its conversions and transforms).
SECTION_OF = {"k_flush": "flush", "k_check": "check", "k_check_final": "check", "k_gen": "generation",
              "k_inject": "injection", "k_xform": "words transform", "k_probe": "probe", "k_sgemm": "fixture"}


def _sections(path):
    text = open(path).read()
    parts = re.split(r"^// -{10,} (.+?)\s*$", text, flags=re.M)
    return {parts[i].strip(): parts[i + 1] for i in range(1, len(parts) - 1, 2)}


def kernel_source_sha(kernel):
    """sha256 of the source that defines `kernel` (short name, e.g. k_flush):
    its section of kernels.hip plus what it uses of the device headers (the
    flush only its streaming stores, the others the whole header; the check
    also the check body's header)."""
    body = _sections(KERNELS_HIP)[SECTION_OF[kernel]]
    if kernel in ("k_check", "k_check_final"):
        body += open(CHECK_HPP).read()
    if kernel == "k_flush":
        body += _sections(DEVICE_HPP)["streaming memory"]
    elif kernel not in ("k_probe", "k_sgemm"):
        body += open(DEVICE_HPP).read()
    return hashlib.sha256(body.encode()).hexdigest()


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def kernel_stats(path):
    out = []
    for r in _rows(path):
        out.append({"name": r["Name"], "calls": int(r["Calls"]), "avg_ns": float(r["AverageNs"]),
                    "min_ns": float(r["MinNs"]), "max_ns": float(r["MaxNs"]), "pct": float(r["Percentage"])})
    return out


def counters(directory, counter):
    """Per-kernel list of per-dispatch values of `counter` from a --pmc run."""
    files = glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError("no counter_collection.csv under %s" % directory)
    per = {}
    for fpath in files:
        for r in _rows(fpath):
            if r.get("Counter_Name") != counter:
                continue
            per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return per


def _short(name):
    return name.split("(")[0].replace("void ", "")


def cmd_stats(a):
    st = kernel_stats(a.csv)
    lines = ["# rocprofv3 kernel trace: %s" % a.title, "", "Command (from the repository root):", "",
             "    " + a.cmd, "", "| Kernel | Calls | Avg (us) | Min (us) | Max (us) | Share |",
             "|---|---|---|---|---|---|"]
    for r in st:
        lines.append("| `%s` | %d | %.2f | %.2f | %.2f | %.2f%% |" % (
            _short(r["name"]), r["calls"], r["avg_ns"] / 1e3, r["min_ns"] / 1e3, r["max_ns"] / 1e3, r["pct"]))
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")


def cmd_select(a):
    """Per-dispatch durations of selected kernels from a kernel-trace CSV:
    each selector is NAME or NAME@GRID (a substring of the kernel name and,
    optionally, the grid size in work-items), so one command's launches can
    be told apart from other launches of the same kernel."""
    rows = _rows(a.trace)
    lines = ["# rocprofv3 kernel trace: %s" % a.title, "", "Command (from the repository root):", "",
             "    " + a.cmd, "", "| Kernel | Grid (work-items) | Dispatches | Median (us) | Mean (us) | Min (us) | Max (us) |",
             "|---|---|---|---|---|---|---|"]
    for sel in a.select:
        name, _, grid = sel.partition("@")
        ds = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows
              if name in r["Kernel_Name"] and (not grid or int(r["Grid_Size_X"]) == int(grid))]
        if not ds:
            lines.append("| `%s` | %s | 0 | - | - | - | - |" % (name, grid or "any"))
            continue
        lines.append("| `%s` | %s | %d | %.2f | %.2f | %.2f | %.2f |" % (
            name, grid or "any", len(ds), statistics.median(ds), statistics.mean(ds), min(ds), max(ds)))
    if a.note:
        lines += ["", a.note]
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")


def kernels_algo():
    """Algorithmic bytes per launch of bench.py --kernels (N = 2^24): a
    generator writes its elements, the injection reads x and writes y, the
    fused generation with injection writes x and y, the two-operand check
    reads both operands and the regenerated-reference check the candidate
    only, the flush writes 1 GiB."""
    N = 1 << 24
    return {
        "krex::k_gen<2, 0, true>": 16 * N * 2, "krex::k_gen<1, 1, false>": N * 2, "krex::k_gen<0, 1, false>": N * 4,
        "krex::k_gen<0, 0, true>": 4 * N * 4, "krex::k_gen<3, 1, false>": 16 * N,
        "krex::k_gen_packed<2, 0, 2>": 16 * N * 2, "krex::k_gen_packed<1, 1, 0>": N * 2,
        "krex::k_gen_packed<3, 0, 2>": 16 * N, "krex::k_gen_packed<3, 1, 0>": 16 * N,
        "krex::k_inject<2, 1>": 16 * N * 4, "krex::k_inject<3, 0>": 16 * N * 2, "krex::k_inject<0, 1>": 4 * N * 8,
        "krex::k_gen_inject<2, 0, true, 1>": 16 * N * 4,
        "krex::k_check<1, 0, true, 2>": N * 6, "krex::k_check<2, 2, true, 3>": 16 * N * 4,
        "krex::k_check<3, 3, true, 3>": 16 * N * 2, "krex::k_check<0, 0, true, 2>": 4 * N * 8,
        "krex::k_check_gen<2, 2, 0, true, true, 2>": 16 * N * 2, "krex::k_check_gen<3, 3, 1, false, true, 2>": 16 * N,
        "krex::k_check_gen<0, 0, 0, true, true, 2>": 4 * N * 4, "krex::k_check_gen<1, 0, 1, false, true, 2>": N * 2,
        "krex::k_check_gen_packed<2, 2, 0, 2, true, 2>": 16 * N * 2,
        "krex::k_check_gen_packed<3, 3, 0, 2, true, 2>": 16 * N,
        "krex::k_flush": 1 << 30,
    }


def default_algo(workload):
    """Algorithmic bytes per launch of the bench command's kernels (the
    generation writes n elements, the check reads both operands, bf16
    candidate and fp32 reference, the flush writes its buffer), or of
    bench.py --kernels."""
    if workload == "kernels":
        return kernels_algo()
    if workload != "gemm_large":
        return {}
    from . import workloads as W
    cfg = W.GEMM_LARGE
    n = cfg["n"] * cfg["n"]
    return {"krex::k_gen<1, 1, false>": n * 2, "krex::k_check<1, 0, true, 2>": n * (2 + 4),
            "krex::k_flush": cfg["flush_bytes"]}


# The launches of bench.py --kernels: what each one is and what bounds it.
KERNEL_ROWS = [
    ("generation, fp32 uniform, 67M", "krex::k_gen<0, 0, true>", "HBM write"),
    ("generation, fp16 uniform, 268M", "krex::k_gen<2, 0, true>", "issue + HBM (Philox word per element)"),
    ("generation, bf16 normal, 16.8M (bench)", "krex::k_gen<1, 1, false>", "vector issue"),
    ("generation, fp32 normal, 16.8M", "krex::k_gen<0, 1, false>", "vector issue"),
    ("generation, fp8 normal, 268M", "krex::k_gen<3, 1, false>", "vector issue"),
    ("packed generation, fp16 uniform, 268M", "krex::k_gen_packed<2, 0, 2>", "HBM write"),
    ("packed generation, bf16 normal, 16.8M", "krex::k_gen_packed<1, 1, 0>", "vector issue"),
    ("packed generation, fp8 uniform, 268M", "krex::k_gen_packed<3, 0, 2>", "HBM write / issue"),
    ("packed generation, fp8 normal, 268M", "krex::k_gen_packed<3, 1, 0>", "vector issue"),
    ("injection, fp16 exact, 268M", "krex::k_inject<2, 1>", "HBM read + write"),
    ("generation + injection in one launch, fp16 uniform exact, 268M", "krex::k_gen_inject<2, 0, true, 1>",
     "vector issue (value + mask word per element)"),
    ("check, bf16 x fp32, 16.8M (bench)", "krex::k_check<1, 0, true, 2>", "HBM read (small launch)"),
    ("check, fp16 x fp16, 268M", "krex::k_check<2, 2, true, 3>", "HBM read"),
    ("check, fp8 x fp8, 268M", "krex::k_check<3, 3, true, 3>", "HBM read (latency: half the time issuing)"),
    ("check, fp32 x fp32, 67M", "krex::k_check<0, 0, true, 2>", "HBM read"),
    ("check vs regenerated reference, fp32 x fp32 uniform, 67M", "krex::k_check_gen<0, 0, 0, true, true, 2>",
     "issue + HBM read (candidate only)"),
    ("check vs regenerated reference, bf16 x fp32 normal, 16.8M", "krex::k_check_gen<1, 0, 1, false, true, 2>",
     "vector issue (normal transform)"),
    ("check vs regenerated reference, fp16 x fp16 uniform, 268M", "krex::k_check_gen<2, 2, 0, true, true, 2>",
     "vector issue (a Philox word per element)"),
    ("check vs regenerated reference, fp8 x fp8 normal, 268M", "krex::k_check_gen<3, 3, 1, false, true, 2>",
     "vector issue (normal transform)"),
    ("check vs regenerated packed reference, fp16 x fp16 uniform, 268M",
     "krex::k_check_gen_packed<2, 2, 0, 2, true, 2>", "vector issue (a Philox block per 8 elements)"),
    ("check vs regenerated packed reference, fp8 x fp8 uniform, 268M",
     "krex::k_check_gen_packed<3, 3, 0, 2, true, 2>", "vector issue (a Philox block per 16 elements)"),
    ("flush, 1 GiB", "krex::k_flush", "HBM write"),
]

HBM_PEAK = 8.0e12


def _own_command():
    """This summarizer's invocation, without its free-text arguments."""
    import sys
    out, skip = [], False
    for x in sys.argv[1:]:
        if skip:
            skip = False
            continue
        if x in ("--cmd", "--note", "--tail", "--title"):
            skip = True
            continue
        out.append(x)
    return "python3 -m paper_2609_30057_amd.profiling " + " ".join(out)


def cmd_throughput(a):
    """Per-kernel throughput of bench.py --kernels from its kernel-trace
    statistics: algorithmic bytes per launch over the average duration."""
    st = {_short(r["name"]): r for r in kernel_stats(a.csv)}
    algo = kernels_algo()
    lines = ["# Per-kernel throughput on the commands' shapes, one MI355X", "",
             "Commands (from the repository root):", "", "    " + a.cmd.replace(" ;; ", "\n    "),
             "    " + _own_command(), ""]
    if a.note:
        lines += [a.note, ""]
    lines += ["| Kernel and shape | Kernel | Time (us) | GB/s | Fraction of 8 TB/s | Bound |",
              "|---|---|---|---|---|---|"]
    for label, k, bound in KERNEL_ROWS:
        r = st.get(k)
        if r is None:
            lines.append("| %s | `%s` | - | - | - | %s |" % (label, k, bound))
            continue
        t = r["avg_ns"] * 1e-9
        bw = algo[k] / t
        lines.append("| %s | `%s` | %.1f | %.0f | %.3f | %s |" % (label, k, t * 1e6, bw / 1e9, bw / HBM_PEAK, bound))
    fin = st.get("krex::k_check_final")
    if fin:
        lines += ["", "`krex::k_check_final` (the check's second launch): %d calls, average %.2f us." % (
            fin["calls"], fin["avg_ns"] / 1e3)]
    if a.tail:
        lines += ["", a.tail]
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")


_DT_SIZE = {0: 4, 1: 2, 2: 2, 3: 1, 4: 4}


def _units(name, algo_bytes):
    """16-byte units of a --kernels launch: one vector of output
    (generation, injection, flush) or of the narrower operand (checks)."""
    m = re.search(r"<(.*)>", name)
    args = [int(x) if x.isdigit() else x for x in (m.group(1).split(", ") if m else [])]
    if "k_check_gen" in name:
        sa, sb = _DT_SIZE[args[0]], _DT_SIZE[args[1]]
        return algo_bytes / sa * min(sa, sb) / 16
    if "k_check<" in name:
        sa, sb = _DT_SIZE[args[0]], _DT_SIZE[args[1]]
        return algo_bytes / (sa + sb) * min(sa, sb) / 16
    if "k_inject" in name or "k_gen_inject" in name:
        return algo_bytes / 32
    return algo_bytes / 16


def cmd_sq(a):
    """SQ counters per kernel from a --pmc run with --kernel-trace (medians
    over each kernel's dispatches at its largest grid)."""
    files = glob.glob(os.path.join(a.dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit("no counter_collection.csv under %s" % a.dir)
    disp = {}
    for fpath in files:
        for r in _rows(fpath):
            key = (fpath, r["Dispatch_Id"])
            d = disp.setdefault(key, {"name": _short(r["Kernel_Name"]), "grid": int(r["Grid_Size"]),
                                      "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
            d[r["Counter_Name"]] = float(r["Counter_Value"])
    per = {}
    for d in disp.values():
        per.setdefault(d["name"], []).append(d)
    algo = kernels_algo()
    lines = ["# SQ counters per kernel (gfx950, one MI355X)", "", "Commands (from the repository root):", "",
             "    " + a.cmd.replace(" ;; ", "\n    "), "    " + _own_command(), ""]
    if a.note:
        lines += [a.note, ""]
    lines += ["| Kernel | us | waves | VALU / wave | SALU / wave | VALU per lane-unit | clock (MHz) | waves/SIMD "
              "| issue-waiting/SIMD |", "|---|---|---|---|---|---|---|---|---|"]
    order = [k for _, k, _ in KERNEL_ROWS] + sorted(k for k in per if k not in [r[1] for r in KERNEL_ROWS])
    med = statistics.median
    for k in order:
        if k not in per:
            continue
        g = max(d["grid"] for d in per[k])
        ds = [d for d in per[k] if d["grid"] == g]
        us = med([d["ns"] for d in ds]) / 1e3
        waves = med([d.get("SQ_WAVES", 0.0) for d in ds])
        valu = med([d.get("SQ_INSTS_VALU", 0.0) for d in ds])
        salu = med([d.get("SQ_INSTS_SALU", 0.0) for d in ds])
        cyc = med([d.get("GRBM_GUI_ACTIVE", 0.0) for d in ds]) / a.xcds
        wc = med([d.get("SQ_WAVE_CYCLES", 0.0) for d in ds])
        wait = med([d.get("SQ_WAIT_INST_ANY", 0.0) for d in ds])
        simds = 4 * a.cus
        per_unit = "%.0f" % (valu * 64 / _units(k, algo[k])) if k in algo else "-"
        lines.append("| `%s` | %.1f | %d | %.0f | %.0f | %s | %.0f | %.1f | %.1f |" % (
            k.replace("krex::", ""), us, waves, valu / max(waves, 1), salu / max(waves, 1), per_unit,
            cyc / (us * 1e-6) / 1e6 if us else 0.0, wc * 4 / (simds * cyc) if cyc else 0.0,
            wait * 4 / (simds * cyc) if cyc else 0.0))
    if a.tail:
        lines += ["", a.tail]
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")


def cmd_traffic(a):
    fetch = counters(a.fetch, "FETCH_SIZE")
    write = counters(a.write, "WRITE_SIZE")
    copy = [k for k in fetch if "copy" in k.lower() or "elementwise" in k.lower()]
    if not copy:
        raise SystemExit("no copy kernel in the counter runs")
    ck = max(copy, key=lambda k: statistics.median(fetch[k]))
    f_copy = statistics.median(fetch[ck]) * 1024.0
    w_copy = statistics.median(write[ck]) * 1024.0
    sf, sw = GIB / f_copy, GIB / w_copy
    algo = json.loads(a.algo) if a.algo else default_algo(a.workload)
    exact = {}
    if a.rdreq:
        parts = {sz: counters(a.rdreq, "TCC_EA0_RDREQ_%dB_sum" % sz) for sz in (32, 64, 128)}
        for k in parts[128]:
            exact[k] = sum(sz * statistics.median(parts[sz].get(k, [0.0])) for sz in (32, 64, 128))
    data = {"calibration": {"kernel": _short(ck), "fetch_bytes": f_copy, "write_bytes": w_copy,
                            "fetch_scale": sf, "write_scale": sw}}
    lines = ["# HBM traffic per dispatch (rocprofv3 FETCH_SIZE / WRITE_SIZE): %s" % a.title, "",
             "Commands (from the repository root):", "", "    " + a.cmd.replace(" ;; ", "\n    "), "",
             "Calibration: `%s`, a plain 1 GiB device copy, reads FETCH %.0f MiB and WRITE %.0f MiB; "
             "scale factors %.4f (fetch) and %.4f (write) turn counter bytes into HBM bytes." % (
                 _short(ck), f_copy / 2**20, w_copy / 2**20, sf, sw), "",
             "| Kernel | Dispatches | FETCH (MiB, scaled) | Read by request size (MiB) | WRITE (MiB, scaled) "
             "| Algorithmic (MiB) | Traffic / algorithmic |",
             "|---|---|---|---|---|---|---|"]
    if a.rdreq:
        cr = exact.get(ck)
        lines[-4] += (" The read-request counters by size give the copy %.1f MiB read (1024 expected)." % (cr / 2**20)
                      if cr else " The copy kernel is missing from the read-request pass.")
    ours = [k for k in fetch if k.startswith(("krex", "void krex"))]
    bases = [_short(k).split("::")[-1].split("<")[0] for k in ours]
    for k in sorted(fetch):
        if not k.startswith(("krex", "void krex")):
            continue
        fb = statistics.median(fetch[k]) * 1024.0 * sf
        wb = statistics.median(write.get(k, [0.0])) * 1024.0 * sw
        rb = exact.get(k)
        key = _short(k)
        al = algo.get(key)
        rd = rb if rb is not None else fb
        lines.append("| `%s` | %d | %.1f | %s | %.1f | %s | %s |" % (
            key, len(fetch[k]), fb / 2**20, "%.1f" % (rb / 2**20) if rb is not None else "-", wb / 2**20,
            "%.1f" % (al / 2**20) if al else "-", "%.3f" % ((rd + wb) / al) if al else "-"))
        fb = rd
        short = key.split("::")[-1].split("<")[0]
        # keyed by the kernel's name, or by its instantiation when the run
        # holds several of one kernel
        name = short if bases.count(short) == 1 else key.split("::")[-1]
        data["%s/%s" % (name, a.workload)] = {
            "kernel": key, "hbm_bytes_per_launch": round(fb + wb), "fetch_bytes": round(fb), "write_bytes": round(wb),
            "algorithmic_bytes": al, "source_sha256": kernel_source_sha(short) if short in SECTION_OF else None}
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    with open(a.out_json, "w") as f:
        json.dump(data, f, indent=1)


def _unit_path(asm, kernel_symbol):
    """Vector instructions of `kernel_symbol`'s per-unit path: from the loop
    head to the first 16-byte store."""
    m = re.search(r"^" + re.escape(kernel_symbol) + r":(.*?)\.Lfunc_end", asm, re.S | re.M)
    if not m:
        raise KeyError(kernel_symbol)
    body = m.group(1).splitlines()
    start = next(i for i, l in enumerate(body) if "Loop Header" in l)
    end = next(i for i, l in enumerate(body) if re.search(r"\b(global|buffer)_store_dwordx4\b", l))
    ops = []
    for l in body[start:end + 1]:
        t = l.strip()
        if t and not t.startswith((".", ";")) and not l.startswith("."):
            ops.append(t.split()[0])
    return [o for o in ops if o.startswith("v_")]


def _op_cost(op, rates):
    base = re.sub(r"_e(32|64)$|_sdwa$|_dpp$", "", op)
    if base in rates:
        return rates[base]
    for prefix, ref in (("v_cmp", "v_cmp_lt_f32"), ("v_cvt_pk_fp8", "v_cvt_pk_fp8_f32"), ("v_cvt_pk_bf16", "v_cvt_pk_bf16_f32"),
                        ("v_cvt_pk_f16", "v_cvt_pk_f16_f32"), ("v_cvt", "v_cvt_f32_u32"), ("v_fmac", "v_fma_f32"),
                        ("v_fmamk", "v_fmaak_f32"), ("v_fma", "v_fma_f32"), ("v_sub_f32", "v_add_f32"),
                        ("v_sub_u32", "v_add_u32"), ("v_add_", "v_add_u32"), ("v_min3", "v_max3_f32"),
                        ("v_min", "v_max_f32"), ("v_max", "v_max_f32"), ("v_or", "v_and_b32"), ("v_xor", "v_and_b32"),
                        ("v_lshl", "v_lshrrev_b32"), ("v_lshr", "v_lshrrev_b32"), ("v_mul_f32", "v_mul_f32"),
                        ("v_mov", "v_and_b32"), ("v_rcp", "v_rcp_f32"), ("v_sqrt", "v_sqrt_f32"),
                        ("v_mad_u64", "v_mad_u64_u32"), ("v_mul_hi", "v_mul_hi_u32"), ("v_perm", "v_perm_b32")):
        if base.startswith(prefix):
            return rates.get(ref, 4.0)
    return 4.0   # unmeasured: the half-rate cost most conversions and 64-bit operations have


PHILOX_PAIR = "philox4x32_10 block (philox_block, two per group)"
PHILOX_LOCKSTEP = "philox4x32_10 block (philox_blocks<2>)"


def philox_mad_cost(rates, name):
    """Issue cost of a v_mad_u64_u32 inside the Philox rounds of kernel
    `name`: its measured block cost less the block's 20 three-way xors, over
    its 20 products (the lockstep form for the word-stream generators and the
    two-block packed units, the compiler's interleaving elsewhere); None
    without the block entries."""
    lock = name.startswith("krex::k_gen<") or name.startswith("krex::k_gen_packed<3, 1")
    key = PHILOX_LOCKSTEP if lock else PHILOX_PAIR
    if key not in rates:
        return None
    return (rates[key] - 20 * _op_cost("v_bitop3_b32", rates)) / 20


def cmd_valu_model(a):
    from paper_2609_30057_amd import build as B
    rates = json.load(open(a.rates))["cycles"]
    asm_path = B.emit_asm(os.path.join(B.BUILD, "kernels.s"))
    asm = open(asm_path).read()
    trace = _rows(a.trace)
    launches = {}
    for r in trace:
        name = _short(r["Kernel_Name"])
        if not name.startswith(("krex::k_gen<", "krex::k_gen_packed<")):
            continue
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        grid = int(r.get("Grid_Size") or r["Grid_Size_X"])
        launches.setdefault(name, []).append((grid, dur))
    clock = 2.4e9
    algo = kernels_algo()
    lines = ["# Vector-issue roofline of the generation kernels: %s" % a.title, "",
             "Commands (from the repository root):", "", "    " + a.cmd.replace(" ;; ", "\n    "), "",
             "Per unit (one thread, one 16-byte output vector) the kernel runs the vector instructions of its "
             "unit path; each costs its measured issue cycles per wave64 instruction (v_fma_f32 = 2). A launch "
             "of u units (its output bytes / 16; a thread may take several) needs u / 64 unit-waves x weighted "
             "cycles / (4 SIMDs x %d CUs x 2.4 GHz) at full vector issue." % a.cus, "",
             "Each unit also writes one 16-byte vector: u x 16 bytes at 8 TB/s is the launch's HBM time. The "
             "larger of the two times bounds the kernel.", "",
             "The rate table prices `v_mad_u64_u32` on its own; inside the Philox rounds each product is read by "
             "the next three-way xor, and the measured Philox block entries put its cost at %s cycles (lockstep "
             "form) and %s cycles (the compiler's interleaving). The last two columns price it so." % (
                 "%.2f" % philox_mad_cost(rates, "krex::k_gen<") if PHILOX_LOCKSTEP in rates else "-",
                 "%.2f" % philox_mad_cost(rates, "x") if PHILOX_PAIR in rates else "-"), "",
             "| Kernel | Vector instr. per unit | Weighted cycles per unit-wave | Unit-waves | Time at full issue (us) "
             "| HBM time (us) | Bound | Measured (us) | Fraction of the bound | Time at full issue, Philox in "
             "context (us) | Fraction of that bound |", "|---|---|---|---|---|---|---|---|---|---|---|"]
    for name in sorted(launches):
        args = re.match(r"krex::k_gen(?:_packed)?<(.*)>", name).group(1).split(", ")
        if "packed" in name:
            sym = "_ZN4krex12k_gen_packedILi%sELi%sELi%sEEEvNS_12PackedParamsE" % tuple(args)
        else:
            sym = "_ZN4krex5k_genILi%sELi%sELb%dEEEvNS_9GenParamsE" % (args[0], args[1], args[2] == "true")
        ops = _unit_path(asm, sym)
        cyc = sum(_op_cost(o, rates) for o in ops)
        mad = philox_mad_cost(rates, name)
        cyc_ctx = None
        if mad is not None:
            ctx = dict(rates, v_mad_u64_u32=mad)
            cyc_ctx = sum(_op_cost(o, ctx) for o in ops)
        grid, _ = max(launches[name])
        durs = [d for g, d in launches[name] if g == grid]
        meas = statistics.median(durs)
        units = algo[name] / 16 if name in algo else grid
        waves = units / 64.0
        t = waves * cyc / (4 * a.cus * clock) * 1e6
        th = units * 16 / 8e12 * 1e6
        tc = waves * cyc_ctx / (4 * a.cus * clock) * 1e6 if cyc_ctx is not None else None
        lines.append("| `%s` | %d | %.0f | %d | %.1f | %.1f | %s | %.1f | %.2f | %s | %s |" % (
            name, len(ops), cyc, waves, t, th, "issue" if t >= th else "HBM", meas, max(t, th) / meas,
            "%.1f" % tc if tc is not None else "-", "%.2f" % (max(tc, th) / meas) if tc is not None else "-"))
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd_name", required=True)
    s = sub.add_parser("stats")
    s.add_argument("--csv", required=True)
    s.add_argument("--out", required=True)
    s.add_argument("--cmd", required=True)
    s.add_argument("--title", default="")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--out-json", required=True)
    t.add_argument("--cmd", required=True)
    t.add_argument("--title", default="")
    t.add_argument("--workload", default="gemm_large")
    t.add_argument("--algo", default="", help="JSON {kernel: algorithmic bytes per launch}")
    t.add_argument("--rdreq", default="", help="directory of the read-request-size counter pass")
    c = sub.add_parser("select")
    c.add_argument("--trace", required=True)
    c.add_argument("--out", required=True)
    c.add_argument("--cmd", required=True)
    c.add_argument("--title", default="")
    c.add_argument("--note", default="")
    c.add_argument("select", nargs="+", help="NAME or NAME@GRID")
    h = sub.add_parser("throughput")
    h.add_argument("--csv", required=True)
    h.add_argument("--out", required=True)
    h.add_argument("--cmd", required=True)
    h.add_argument("--note", default="")
    h.add_argument("--tail", default="")
    q = sub.add_parser("sq")
    q.add_argument("--dir", required=True)
    q.add_argument("--out", required=True)
    q.add_argument("--cmd", required=True)
    q.add_argument("--note", default="")
    q.add_argument("--tail", default="")
    q.add_argument("--cus", type=int, default=256)
    q.add_argument("--xcds", type=int, default=8)
    v = sub.add_parser("valu-model")
    v.add_argument("--rates", required=True)
    v.add_argument("--trace", required=True)
    v.add_argument("--out", required=True)
    v.add_argument("--cmd", required=True)
    v.add_argument("--title", default="")
    v.add_argument("--cus", type=int, default=256)
    a = ap.parse_args()
    if a.cmd_name == "stats":
        cmd_stats(a)
    elif a.cmd_name == "traffic":
        cmd_traffic(a)
    elif a.cmd_name == "select":
        cmd_select(a)
    elif a.cmd_name == "throughput":
        cmd_throughput(a)
    elif a.cmd_name == "sq":
        cmd_sq(a)
    else:
        cmd_valu_model(a)


if __name__ == "__main__":
    main()
