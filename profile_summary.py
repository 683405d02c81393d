"""Summaries of rocprofv3 output for profiles/ (reads CSV files, runs nothing).

  python profile_summary.py stats  <kernel_stats.csv> <out.md> <command...>
      per-kernel calls / average / total time of the library's kernels.

  python profile_summary.py traffic <fetch_dir> <write_dir> <workload> <out.md> <command...>
      HBM bytes per dispatch of each phase's kernel from two `--pmc` runs
      (FETCH_SIZE, then WRITE_SIZE; both in KiB per dispatch), each scaled by
      what the same counter reads for the plain 1 GiB copy that
      `bench.py --copy-calibration` runs first (a torch `neg` kernel: reads
      1 GiB, writes 1 GiB). Updates profiles/hbm_traffic.json, which bench.py
      reads for roofline.traffic while the kernel source is unchanged.
"""

from __future__ import annotations

import csv
import glob
import json
import os
import re
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

COPY_BYTES = 1 << 30
# Kernel of each phase (first match of the demangled name).
PHASE_KERNELS = {
    "qstats": r"jacap::qstats_kernel",
    "kpass": r"jacap::kpass_kernel",
    "weights": r"jacap::softmax_weights_kernel",
    "gram": r"jacap::gram_mfma_kernel<\d+, 2>",
    "leverage": r"jacap::leverage_mfma_kernel",
    "select": r"jacap::select_kernel",
    "compact": r"jacap::compact_kernel",
}


def stats(csv_path, out_md, command):
    rows = list(csv.DictReader(open(csv_path)))
    rows = [r for r in rows if "jacap::" in r["Name"]]
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = ["| kernel | calls | avg us | min us | max us | share |", "|---|---:|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = r["Name"].split("(")[0].replace("void ", "")
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{100 * float(r['TotalDurationNs']) / total:.1f}% |")
    with open(out_md, "w") as fh:
        fh.write("# rocprofv3 kernel statistics\n\nCommand:\n\n```\n" + command + "\n```\n\n")
        fh.write("\n".join(lines) + "\n")


def _per_dispatch(pmc_dir, counter):
    """[(kernel name, value)] per dispatch, in dispatch order."""
    files = glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {pmc_dir}")
    vals = defaultdict(float)
    names = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r.get("Counter_Name") != counter:
                continue
            key = int(r["Dispatch_Id"])
            vals[key] += float(r["Counter_Value"])
            names[key] = r["Kernel_Name"]
    return [(names[k], vals[k]) for k in sorted(vals)]


def traffic(fetch_dir, write_dir, workload, out_md, command):
    import bench  # for source_sha (bench does not touch the GPU on import)

    fetch = _per_dispatch(fetch_dir, "FETCH_SIZE")
    write = _per_dispatch(write_dir, "WRITE_SIZE")

    def calib(disp):
        cands = [(n, v) for n, v in disp if re.search(r"neg", n, re.I)]
        if not cands:
            raise SystemExit("calibration copy (neg kernel) not found")
        n, v = max(cands, key=lambda nv: nv[1])
        return n, COPY_BYTES / (v * 1024.0)

    cf_name, cf = calib(fetch)
    cw_name, cw = calib(write)
    try:
        rec = json.load(open(bench.TRAFFIC_FILE))
    except (OSError, ValueError):
        rec = {}
    lines = ["| phase | kernel | dispatches | FETCH KiB | WRITE KiB | HBM bytes / launch |",
             "|---|---|---:|---:|---:|---:|"]
    for phase, pat in PHASE_KERNELS.items():
        fv = [v for n, v in fetch if re.search(pat, n)]
        wv = [v for n, v in write if re.search(pat, n)]
        if not fv or not wv:
            continue
        f_kib, w_kib = sum(fv) / len(fv), sum(wv) / len(wv)
        fb, wb = f_kib * 1024 * cf, w_kib * 1024 * cw
        rec[phase] = {"workload": workload, "source_sha": bench.source_sha(phase),
                      "kernel": pat, "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                      "hbm_bytes_per_launch": fb + wb, "dispatches": len(fv),
                      "fetch_scale": cf, "write_scale": cw}
        lines.append(f"| {phase} | `{pat}` | {len(fv)} | {f_kib:.0f} | {w_kib:.0f} | {fb + wb:.4g} |")
    with open(bench.TRAFFIC_FILE, "w") as fh:
        json.dump(rec, fh, indent=1, sort_keys=True)
    with open(out_md, "w") as fh:
        fh.write(f"# HBM traffic per dispatch ({workload})\n\nCommand:\n\n```\n{command}\n```\n\n")
        fh.write(f"Calibration: a 1 GiB copy ({cf_name.split('(')[0][:80]}) reads "
                 f"FETCH_SIZE x {cf:.4f} and WRITE_SIZE x {cw:.4f} of its true bytes.\n\n")
        fh.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    mode = sys.argv[1]
    if mode == "stats":
        stats(sys.argv[2], sys.argv[3], " ".join(sys.argv[4:]))
    elif mode == "traffic":
        traffic(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5], " ".join(sys.argv[6:]))
    else:
        raise SystemExit(__doc__)
