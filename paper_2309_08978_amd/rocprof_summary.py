"""Summarise a rocprofv3 run of bench.py for the profiles/ folder.

Reads the CSV outputs of ``rocprofv3 --kernel-trace --stats -f csv`` (the
``*_kernel_stats.csv`` summary and the ``*_kernel_trace.csv`` dispatch list)
or of a ``--pmc`` run (``*_counter_collection.csv``), and prints:

* rocprofv3's own per-kernel statistics (all dispatches of a kernel symbol);
* per (kernel symbol, grid) statistics over the last ``--last`` dispatches,
  which is the timed region of bench.py (a kernel instance that serves two
  shapes is listed once per grid);
* for a counter run, the per-dispatch mean of each counter per (kernel, grid).

    python -m paper_2309_08978_amd.rocprof_summary <rocprofv3 output dir> [--last N]
"""
from __future__ import annotations

import argparse
import csv
import glob
import os
import statistics
import sys
from collections import OrderedDict


def _short(name: str) -> str:
    name = name.replace("void nnjit::", "").replace("nnjit::", "")
    return name.split("(")[0]


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def summarize(out_dir: str, last: int, top: int = 12) -> str:
    lines = []
    stats = sorted(glob.glob(os.path.join(out_dir, "**", "*kernel_stats.csv"), recursive=True))
    trace = sorted(glob.glob(os.path.join(out_dir, "**", "*kernel_trace.csv"), recursive=True))
    pmc = sorted(glob.glob(os.path.join(out_dir, "**", "*counter_collection.csv"), recursive=True))
    if stats:
        rows = _rows(stats[0])
        lines.append(f"rocprofv3 --stats ({os.path.basename(stats[0])}), top {top} by total time:")
        lines.append(f"  {'kernel':62s} {'calls':>6s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} {'pct':>6s}")
        for r in rows[:top]:
            lines.append(f"  {_short(r['Name'])[:62]:62s} {int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:9.2f} "
                         f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f} {float(r['Percentage']):6.2f}")
    if trace:
        rows = _rows(trace[0])
        rows.sort(key=lambda r: int(r["Start_Timestamp"]))
        sel = rows[-last:] if last > 0 else rows
        groups = OrderedDict()
        for r in sel:
            wg = int(r.get("Workgroup_Size_X", r.get("Workgroup_Size", 1)) or 1)
            grid = (int(r["Grid_Size_X"]) // max(wg, 1), int(r.get("Grid_Size_Z", 1) or 1))
            key = (_short(r["Kernel_Name"]), grid)
            groups.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        lines.append("")
        lines.append(f"per (kernel, grid) over the last {len(sel)} dispatches (the timed region):")
        lines.append(f"  {'kernel':62s} {'WGs':>6s} {'z':>4s} {'n':>5s} {'mean_us':>9s} {'median_us':>9s} {'min_us':>8s}")
        for (k, (gx, gz)), d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
            lines.append(f"  {k[:62]:62s} {gx:6d} {gz:4d} {len(d):5d} {statistics.mean(d):9.2f} "
                         f"{statistics.median(d):9.2f} {min(d):8.2f}")
    if pmc:
        rows = _rows(pmc[0])
        groups = OrderedDict()
        for r in rows:
            wg = int(r.get("Workgroup_Size", 1) or 1)
            key = (_short(r["Kernel_Name"]), int(r.get("Grid_Size", 0) or 0) // max(wg, 1), r["Counter_Name"])
            groups.setdefault(key, {}).setdefault(r.get("Dispatch_Id", len(groups)), 0.0)
            groups[key][r.get("Dispatch_Id")] += float(r["Counter_Value"])
        lines.append("")
        lines.append("counters, mean per dispatch per (kernel, WGs):")
        for (k, g, c), per in groups.items():
            vals = list(per.values())
            lines.append(f"  {k[:62]:62s} {g:6d} {c:14s} n={len(vals):4d} mean={statistics.mean(vals):.1f}")
    if not lines:
        lines.append(f"no rocprofv3 CSV output found under {out_dir}")
    return "\n".join(lines)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("out_dir")
    ap.add_argument("--last", type=int, default=0, help="only the last N dispatches in the per-grid table")
    ap.add_argument("--top", type=int, default=12)
    a = ap.parse_args(argv)
    print(summarize(a.out_dir, a.last, a.top))
    return 0


if __name__ == "__main__":
    sys.exit(main())
