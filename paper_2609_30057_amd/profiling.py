"""Summaries of rocprofv3 output (CSV) for the committed profiles.

  python -m paper_2609_30057_amd.profiling stats  --csv DIR/..._kernel_stats.csv --out FILE.md --cmd "..."
  python -m paper_2609_30057_amd.profiling traffic --fetch DIR --write DIR --out-json profiles/traffic.json
                                                 --out FILE.md --cmd "..."

traffic: per-dispatch FETCH_SIZE and WRITE_SIZE (KiB) of each kernel, scaled by
what the same counters read for a plain device copy of 1 GiB (1 GiB fetched,
1 GiB written), and compared with the kernel's algorithmic bytes.
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

# kernels.hip is split into sections by "// ---- <name>" rules; a traffic
# figure is tied to the source of its kernel's section (plus the device
# header for the kernels that use its conversions and transforms).
SECTION_OF = {"k_flush": "flush", "k_check": "check", "k_check_final": "check", "k_gen": "generation",
              "k_inject": "injection", "k_xform": "words transform", "k_probe": "probe", "k_sgemm": "fixture"}


def kernel_source_sha(kernel):
    """sha256 of the source that defines `kernel` (short name, e.g. k_flush)."""
    text = open(KERNELS_HIP).read()
    parts = re.split(r"^// -{10,} (.+?)\s*$", text, flags=re.M)
    sections = {parts[i].strip(): parts[i + 1] for i in range(1, len(parts) - 1, 2)}
    body = sections[SECTION_OF[kernel]]
    if kernel not in ("k_flush", "k_probe", "k_sgemm"):
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
    algo = json.loads(a.algo) if a.algo else {}
    data = {"calibration": {"kernel": _short(ck), "fetch_bytes": f_copy, "write_bytes": w_copy,
                            "fetch_scale": sf, "write_scale": sw}}
    lines = ["# HBM traffic per dispatch (rocprofv3 FETCH_SIZE / WRITE_SIZE): %s" % a.title, "",
             "Commands (from the repository root):", "", "    " + a.cmd.replace(" ;; ", "\n    "), "",
             "Calibration: `%s`, a plain 1 GiB device copy, reads FETCH %.0f MiB and WRITE %.0f MiB; "
             "scale factors %.4f (fetch) and %.4f (write) turn counter bytes into HBM bytes." % (
                 _short(ck), f_copy / 2**20, w_copy / 2**20, sf, sw), "",
             "| Kernel | Dispatches | FETCH (MiB, scaled) | WRITE (MiB, scaled) | Algorithmic (MiB) | Traffic / algorithmic |",
             "|---|---|---|---|---|---|"]
    for k in sorted(fetch):
        if not k.startswith(("krex", "void krex")):
            continue
        fb = statistics.median(fetch[k]) * 1024.0 * sf
        wb = statistics.median(write.get(k, [0.0])) * 1024.0 * sw
        key = _short(k)
        al = algo.get(key)
        lines.append("| `%s` | %d | %.1f | %.1f | %s | %s |" % (
            key, len(fetch[k]), fb / 2**20, wb / 2**20, "%.1f" % (al / 2**20) if al else "-",
            "%.3f" % ((fb + wb) / al) if al else "-"))
        short = key.split("::")[-1].split("<")[0]
        data["%s/%s" % (short, a.workload)] = {
            "kernel": key, "hbm_bytes_per_launch": round(fb + wb), "fetch_bytes": round(fb), "write_bytes": round(wb),
            "algorithmic_bytes": al, "source_sha256": kernel_source_sha(short) if short in SECTION_OF else None}
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    with open(a.out_json, "w") as f:
        json.dump(data, f, indent=1)


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
    a = ap.parse_args()
    if a.cmd_name == "stats":
        cmd_stats(a)
    else:
        cmd_traffic(a)


if __name__ == "__main__":
    main()
