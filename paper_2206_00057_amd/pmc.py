"""Text summaries of rocprofv3 output for the kernels of libdigest.so.

Kernel durations (from a ``rocprofv3 --kernel-trace --stats`` run):

    python -m paper_2206_00057_amd.pmc stats --csv <dir>/<name>_kernel_stats.csv \\
        --title "..." --command "..." --out profiles/<kernel-or-workload>_kernel_stats.txt

L2-to-fabric traffic of one kernel (the bytes its L2 misses move between the
L2s and the memory side, Infinity Cache hits included; not HBM bytes alone),
from two counter passes over the same command:

    python -m paper_2206_00057_amd.pmc traffic \\
        --fetch <fetch-dir>/fetch_counter_collection.csv \\
        --write <write-dir>/write_counter_collection.csv \\
        --kernel-name "k_gemm<64, 64, true, false, false, true" --key gemm_dw_splitk.l1 \\
        --copy-bytes 268435456 --workload medium --out profiles/medium_hbm_traffic.txt

Per-kernel counter averages from one counter pass (e.g. MFMA utilisation):

    python -m paper_2206_00057_amd.pmc counters --csv <dir>/<name>_counter_collection.csv \
        --kernel-name "k_gemm<64, 64" --title "..." --command "..." --out profiles/<name>.txt

FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the kernel's dispatches are
averaged, then each is divided by what the same counter reads, per byte, for
a plain copy kernel of known size (the largest "copyBuffer" dispatch of the
run, a device-to-device copy of --copy-bytes bytes).  The summary records the
hash of the kernel sources; bench.py reports the figure only while that hash
still matches.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def kernel_source_hash() -> str:
    """Hash of the sources that define the kernels and their launches."""
    h = hashlib.sha256()
    for f in ("digest_kernels.hip", "kernels.h", "digest_host.cpp"):
        with open(os.path.join(ROOT, "paper_2206_00057_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _rows(path, counter):
    out = []
    with open(path) as fh:
        for r in csv.DictReader(fh):
            if r.get("Counter_Name", counter) == counter:
                out.append((r["Kernel_Name"], float(r["Counter_Value"]), int(r["Grid_Size"])))
    return out


def _pick(rows, kernel_name, grid_size=0, largest_grid=False):
    """Counter values of the dispatches of one kernel: those whose name
    contains kernel_name, and of those the ones of one launch shape (a grid
    of grid_size work-items, or the largest grid among them) when asked."""
    m = [(v, g) for n, v, g in rows if kernel_name in n]
    if grid_size:
        m = [(v, g) for v, g in m if g == grid_size]
    elif largest_grid and m:
        top = max(g for _, g in m)
        m = [(v, g) for v, g in m if g == top]
    return [v for v, _ in m]


def summarize(fetch_csv, write_csv, kernel_name, copy_name, copy_bytes, grid_size=0,
              largest_grid=False):
    f = _rows(fetch_csv, "FETCH_SIZE")
    w = _rows(write_csv, "WRITE_SIZE")
    kf = _pick(f, kernel_name, grid_size, largest_grid)
    kw = _pick(w, kernel_name, grid_size, largest_grid)
    cf = max(v for n, v, _ in f if copy_name in n)
    cw = max(v for n, v, _ in w if copy_name in n)
    if not kf or not kw:
        raise SystemExit(f"no dispatch of {kernel_name!r} in the counter files")
    fetch_kib = sum(kf) / len(kf)
    write_kib = sum(kw) / len(kw)
    fetch_scale = cf * 1024.0 / copy_bytes
    write_scale = cw * 1024.0 / copy_bytes
    traffic = fetch_kib * 1024.0 / fetch_scale + write_kib * 1024.0 / write_scale
    names = sorted({n for n, _, _ in f if kernel_name in n})
    return {
        "rocprof_kernel": names[0] if names else kernel_name,
        "dispatches": len(kf),
        "fetch_kib_per_dispatch": round(fetch_kib, 1),
        "write_kib_per_dispatch": round(write_kib, 1),
        "calibration_copy_bytes": copy_bytes,
        "calibration_fetch_kib": round(cf, 1),
        "calibration_write_kib": round(cw, 1),
        "fetch_scale": round(fetch_scale, 4),
        "write_scale": round(write_scale, 4),
        "traffic_bytes_per_launch": round(traffic),
    }


def counters_table(path, patterns):
    """Average of every counter over the dispatches of each kernel whose name
    contains one of the patterns, as fixed-width text."""
    per = {}
    with open(path) as fh:
        for r in csv.DictReader(fh):
            name = r["Kernel_Name"]
            if not any(p in name for p in patterns):
                continue
            name = re.sub(r"\(anonymous namespace\)::", "", name)
            name = re.sub(r"\((.*)\)$", "", name).replace("void ", "")
            d = per.setdefault(name, {})
            d.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            d.setdefault("_ns", {})[r["Dispatch_Id"]] = (int(r["End_Timestamp"]) -
                                                        int(r["Start_Timestamp"]))
    out = []
    for name, d in per.items():
        ns = d.pop("_ns")
        avg = {k: sum(v) / len(v) for k, v in d.items()}
        out.append(f"{name}: {len(ns)} dispatches, {sum(ns.values()) / len(ns) / 1e3:.2f} us "
                   "per dispatch")
        for k in sorted(avg):
            out.append(f"  {k:32s} {avg[k]:16.1f}")
        if "SQ_INSTS_MFMA" in avg and "SQ_VALU_MFMA_BUSY_CYCLES" in avg and avg["SQ_INSTS_MFMA"]:
            out.append(f"  {'busy cycles per MFMA':32s} "
                       f"{avg['SQ_VALU_MFMA_BUSY_CYCLES'] / avg['SQ_INSTS_MFMA']:16.1f}")
        if "SQ_WAIT_INST_ANY" in avg and avg.get("SQ_WAVE_CYCLES"):
            out.append(f"  {'dependency-wait share of wave time':32s} "
                       f"{avg['SQ_WAIT_INST_ANY'] / avg['SQ_WAVE_CYCLES']:16.3f}")
    return out


def stats_table(path):
    """Per-kernel rows of a rocprofv3 kernel_stats.csv, as fixed-width text."""
    out = [f"# {'kernel':70s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} "
           f"{'total_ms':>9s} {'pct':>6s}"]
    with open(path) as fh:
        for r in csv.DictReader(fh):
            name = re.sub(r"\(anonymous namespace\)::", "", r["Name"])
            name = re.sub(r"\((.*)\)$", "", name).replace("void ", "")
            out.append(f"  {name[:70]:70s} {r['Calls']:>6s} {float(r['AverageNs']) / 1e3:9.2f} "
                       f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f} "
                       f"{float(r['TotalDurationNs']) / 1e6:9.3f} {float(r['Percentage']):6.2f}")
    return out


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    st = sub.add_parser("stats", help="format a kernel_stats.csv")
    st.add_argument("--csv", required=True)
    st.add_argument("--title", required=True)
    st.add_argument("--command", action="append", default=[])
    st.add_argument("--out", required=True)
    co = sub.add_parser("counters", help="per-kernel averages of a counter pass")
    co.add_argument("--csv", required=True)
    co.add_argument("--kernel-name", action="append", required=True,
                    help="substring of the rocprof kernel names to include (repeatable)")
    co.add_argument("--title", required=True)
    co.add_argument("--command", action="append", default=[])
    co.add_argument("--out", required=True)
    tr = sub.add_parser("traffic", help="L2-fabric bytes per launch of one kernel")
    tr.add_argument("--fetch", required=True)
    tr.add_argument("--write", required=True)
    tr.add_argument("--kernel-name", required=True, help="substring of the rocprof kernel name")
    tr.add_argument("--key", required=True, help="bench.py kernel key, e.g. gemm_dw_splitk.l1")
    tr.add_argument("--grid-size", type=int, default=0,
                    help="only the dispatches of this grid (work-items), e.g. one layer's launch")
    tr.add_argument("--largest-grid", action="store_true",
                    help="only the dispatches of the largest grid among the matches")
    tr.add_argument("--copy-name", default="copyBuffer")
    tr.add_argument("--copy-bytes", type=int, required=True)
    tr.add_argument("--workload", required=True)
    tr.add_argument("--command", action="append", default=[])
    tr.add_argument("--out", required=True)
    a = ap.parse_args()
    if a.cmd == "stats":
        lines = [f"# {a.title}"] + [f"# command: {c}" for c in a.command]
        lines += [f"# source: rocprofv3 --kernel-trace --stats ({os.path.basename(a.csv)})", "#"]
        lines += stats_table(a.csv)
    elif a.cmd == "counters":
        lines = [f"# {a.title}"] + [f"# command: {c}" for c in a.command]
        lines += [f"# source: rocprofv3 --pmc ({os.path.basename(a.csv)})",
                  f"# source_sha = {kernel_source_hash()}", "#"]
        lines += counters_table(a.csv, a.kernel_name)
    else:
        s = summarize(a.fetch, a.write, a.kernel_name, a.copy_name, a.copy_bytes, a.grid_size,
                      a.largest_grid)
        lines = [f"# L2-to-fabric traffic of one launch of {a.key} on the {a.workload} workload:",
                 "# the bytes the L2s of the 8 XCDs request from and write to the memory side",
                 "# (Infinity Cache hits included, so not HBM bytes alone), from rocprofv3",
                 "# FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by the counter's",
                 "# reading per byte of a plain device-to-device copy of known size.",
                 "# commands:"]
        lines += [f"#   {c}" for c in a.command]
        lines += [f"kernel = {a.key}", f"source_sha = {kernel_source_hash()}"]
        lines += [f"{k} = {v}" for k, v in s.items()]
    with open(a.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
