"""Summaries of rocprofv3 output for profiles/ (reads CSV files, runs nothing).

  python profile_summary.py stats  <kernel_stats.csv> <out.md> <command...>
      per-kernel calls / average / total time of the library's kernels.

  python profile_summary.py sq <out.md> <command> <pmc_dir>...
      per-kernel utilisation and stall fractions from `--pmc` runs of SQ
      counters (first dispatch of each library kernel; any of the counters
      below that the runs collected).

  python profile_summary.py traffic|traffic-summary <fetch_dir> <write_dir> <workload> <out.md> <command...>
      HBM bytes per dispatch of each phase's kernel from two `--pmc` runs
      (FETCH_SIZE, then WRITE_SIZE; both in KiB per dispatch), each scaled by
      what the same counter reads for the plain 1 GiB copy that
      `bench.py --copy-calibration` runs first (a torch `neg` kernel: reads
      1 GiB, writes 1 GiB). Updates profiles/hbm_traffic.json, which bench.py
      reads for roofline.traffic while the kernel source is unchanged
      (traffic-summary: the summary only, profiles/hbm_traffic.json untouched).
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
    "kpass": r"jacap::kpass_(quad_)?kernel",
    "kpass_tri": r"jacap::kpass_tri_kernel",
    "qfactor": r"jacap::qfactor_kernel",
    "weights": r"jacap::softmax_weights_kernel",
    "gram": r"jacap::gram_mfma_kernel<\d+, 2, \d+>",
    "leverage": r"jacap::leverage_mfma_kernel",
    "select": r"jacap::select_kernel",
    "compact": r"jacap::compact_kernel",
}


def _kernel_name(full):
    return full.replace("(anonymous namespace)::", "").split("(")[0].replace("void ", "")


def stats(csv_path, out_md, command):
    rows = list(csv.DictReader(open(csv_path)))
    rows = [r for r in rows if "jacap::" in r["Name"]]
    # the streaming-read probe that bench.py runs after its timed region is
    # not part of the path: listed apart, outside the shares
    probe = [r for r in rows if "stream_read_kernel" in r["Name"]]
    rows = [r for r in rows if "stream_read_kernel" not in r["Name"]]
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = ["| kernel | calls | avg us | min us | max us | share |", "|---|---:|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append(f"| `{_kernel_name(r['Name'])}` | {r['Calls']} | "
                     f"{float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{100 * float(r['TotalDurationNs']) / total:.1f}% |")
    for r in probe:
        lines.append(f"\nRead probe (not part of the path): `{_kernel_name(r['Name'])}`, "
                     f"{r['Calls']} calls, {float(r['AverageNs']) / 1e3:.1f} us average.")
    with open(out_md, "w") as fh:
        fh.write("# rocprofv3 kernel statistics\n\nCommand:\n\n```\n" + command + "\n```\n\n")
        fh.write("\n".join(lines) + "\n")


def _first_dispatch_counters(pmc_dirs):
    """{kernel: {counter: value}} for the first dispatch of each jacap kernel.
    Rows of one run are summed (one per XCD or instance); a counter that
    several runs collected (GRBM_GUI_ACTIVE) is taken from the first."""
    vals = defaultdict(dict)
    for d in pmc_dirs:
        run = defaultdict(dict)
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            first = {}
            for r in csv.DictReader(open(f)):
                if "jacap::" not in r["Kernel_Name"]:
                    continue
                name = _kernel_name(r["Kernel_Name"])
                did = int(r["Dispatch_Id"])
                if first.setdefault(name, did) != did:
                    continue
                c = r["Counter_Name"]
                run[name][c] = run[name].get(c, 0.0) + float(r["Counter_Value"])
        for name, cs in run.items():
            for c, v in cs.items():
                vals[name].setdefault(c, v)
    return vals


def sq(out_md, command, pmc_dirs):
    """Fractions per kernel. GRBM_GUI_ACTIVE is summed over the 8 XCDs, so
    GUI/8 is the kernel's cycles; per-SIMD rates divide by 1024 SIMDs, per-CU
    rates by 256 CUs; wave fractions divide by SQ_WAVE_CYCLES."""
    vals = _first_dispatch_counters(pmc_dirs)
    cols = [
        ("MFMA busy", lambda v, cyc: v["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * 1024)),
        ("VALU active", lambda v, cyc: v["SQ_ACTIVE_INST_VALU"] / (cyc * 256)),
        ("LDS active", lambda v, cyc: v["SQ_ACTIVE_INST_LDS"] / (cyc * 256)),
        ("LDS bank conflict", lambda v, cyc: v["SQ_LDS_BANK_CONFLICT"] / v["SQ_LDS_IDX_ACTIVE"]),
        ("wave: waiting on data", lambda v, cyc: v["SQ_WAIT_ANY"] / v["SQ_WAVE_CYCLES"]),
        ("wave: ready, not issued", lambda v, cyc: v["SQ_WAIT_INST_ANY"] / v["SQ_WAVE_CYCLES"]),
        ("wave: issuing", lambda v, cyc: v["SQ_ACTIVE_INST_ANY"] / v["SQ_WAVE_CYCLES"]),
        ("MFMA-VALU co-exec", lambda v, cyc: v["SQ_VALU_MFMA_COEXEC_CYCLES"] / (cyc * 1024)),
        ("L2 hit", lambda v, cyc: v["TCC_HIT_sum"] / (v["TCC_HIT_sum"] + v["TCC_MISS_sum"])),
    ]
    names = [c for c, f in cols if any(_ok(f, v) for v in vals.values())]
    lines = ["| kernel | " + " | ".join(names) + " |", "|---|" + "---:|" * len(names)]
    for k, v in vals.items():
        cyc = v.get("GRBM_GUI_ACTIVE", 8.0) / 8.0
        row = []
        for c, f in cols:
            if c not in names:
                continue
            x = _ok(f, v, cyc)
            row.append("" if x is None else f"{100 * x:.1f}%")
        lines.append(f"| `{k}` | " + " | ".join(row) + " |")
    with open(out_md, "w") as fh:
        fh.write("# SQ counters per kernel (first dispatch of each)\n\nCommand (one run per "
                 "counter set):\n\n```\n" + command + "\n```\n\n" + (sq.__doc__ or "")
                 .replace("\n    ", " ").strip() + "\n\n")
        fh.write("\n".join(lines) + "\n")


def _ok(f, v, cyc=None):
    try:
        return f(v, v.get("GRBM_GUI_ACTIVE", 8.0) / 8.0 if cyc is None else cyc)
    except (KeyError, ZeroDivisionError):
        return None


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


def traffic(fetch_dir, write_dir, workload, out_md, command, record=True):
    """record=False writes the summary only (a workload other than the one
    bench.py's default line reports)."""
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
    if record:
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
    elif mode == "sq":
        sq(sys.argv[2], sys.argv[3], sys.argv[4:])
    elif mode in ("traffic", "traffic-summary"):
        traffic(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5], " ".join(sys.argv[6:]),
                record=mode == "traffic")
    else:
        raise SystemExit(__doc__)
