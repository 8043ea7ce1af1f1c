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

With --traffic FETCH_DIR WRITE_DIR --meta META [--db profiles/traffic.json] it
turns two counter runs of ``bench.py --profile-op`` (``rocprofv3 --pmc
FETCH_SIZE`` and ``--pmc WRITE_SIZE``) into HBM bytes per launch of the
profiled product, scaled by the reference copy in the same run.  With
--mfma PMC_DIR --meta META it reports the matrix-core busy fraction of the
product from a ``--pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE ...`` run.
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


def _pmc_dispatches(out_dir, counter):
    """[(kernel name, grid in workgroups, counter value)] in dispatch order."""
    path = sorted(glob.glob(os.path.join(out_dir, "**", "*counter_collection.csv"), recursive=True))
    if not path:
        raise SystemExit(f"no counter_collection.csv under {out_dir}")
    per = OrderedDict()
    for r in _rows(path[0]):
        if r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        wg = int(r.get("Workgroup_Size", 1) or 1)
        if d not in per:
            per[d] = [r["Kernel_Name"], int(r.get("Grid_Size", 0) or 0) // max(wg, 1), 0.0]
        per[d][2] += float(r["Counter_Value"])
    return [tuple(v) for _, v in sorted(per.items())]


def traffic(fetch_dir, write_dir, meta):
    """HBM bytes per launch of the profiled product (bench.py --profile-op):
    the product's dispatches after the reference copy, FETCH_SIZE and
    WRITE_SIZE (KiB) each scaled by what the counter reads for the copy."""
    ref_bytes = meta["copy_ref_mb"] << 20
    out = {}
    for key, d, counter in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        rows = _pmc_dispatches(d, counter)
        is_copy = lambda r: "copyBuffer" in r[0] or "copy_kernel" in r[0]
        copies = [i for i, r in enumerate(rows) if is_copy(r)]
        if not copies:
            raise SystemExit(f"{d}: no reference copy dispatch found")
        # the reference is the run of same-grid copies right before the
        # product's launches (other copies, e.g. operand clones, may precede)
        ref_ids = [copies[-1]]
        while ref_ids[0] > 0 and is_copy(rows[ref_ids[0] - 1]) and rows[ref_ids[0] - 1][1] == rows[copies[-1]][1]:
            ref_ids.insert(0, ref_ids[0] - 1)
        ref = statistics.mean(rows[i][2] for i in ref_ids)
        factor = ref_bytes / (ref * 1024.0)
        after = [r for r in rows[copies[-1] + 1:] if "nnjit" in r[0]]
        kib = sum(r[2] for r in after) / meta["reps"]
        out[key] = {"kib_per_launch_raw": round(kib, 1), "scale": round(factor, 4),
                    "bytes_per_launch": round(kib * 1024.0 * factor),
                    "kernels": sorted({f"{_short(r[0])} x{r[1]}" for r in after})}
    total = out["fetch"]["bytes_per_launch"] + out["write"]["bytes_per_launch"]
    return {"digest": meta["digest"], "hbm_bytes_per_launch": total, "algorithmic_bytes": meta["algorithmic_bytes"],
            "ratio_to_algorithmic": round(total / meta["algorithmic_bytes"], 3), "fetch": out["fetch"],
            "write": out["write"], "reps": meta["reps"], "copy_ref_mb": meta["copy_ref_mb"]}


def kernel_duration_us(trace_dir, steady_n: int = 20):
    """Durations (us) of the profiled product's dispatches in a --kernel-trace
    run of bench.py --profile-op: the mean over the library's dispatches
    after the last reference copy (the counted launches), the mean over the
    last `steady_n` dispatches of the same kernels before the copies (the
    half-second warm-up: the clock and caches of the timed steps; the copies
    themselves disturb the first launches after them), and the kernel names."""
    path = sorted(glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True))
    if not path:
        raise SystemExit(f"no kernel_trace.csv under {trace_dir}")
    rows = sorted(_rows(path[0]), key=lambda r: int(r["Start_Timestamp"]))
    is_copy = lambda r: "copyBuffer" in r["Kernel_Name"] or "copy_kernel" in r["Kernel_Name"]
    copies = [i for i, r in enumerate(rows) if is_copy(r)]
    last = copies[-1] if copies else -1
    after = [r for r in rows[last + 1:] if "nnjit" in r["Kernel_Name"]]
    if not after:
        return None, None, []
    names = {r["Kernel_Name"] for r in after}
    first_ref = last
    while first_ref > 0 and is_copy(rows[first_ref - 1]):
        first_ref -= 1
    before = [r for r in rows[:max(first_ref, 0)] if r["Kernel_Name"] in names][-steady_n:]
    dur = lambda rs: statistics.mean((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rs)
    return dur(after), (dur(before) if before else None), sorted({_short(n) for n in names})


def mfma_busy(pmc_dir, meta, simds: int = 1024, trace_dir=None, clock_ghz: float = 2.4):
    """Matrix-core busy fraction of the profiled product from one counter run
    of SQ_VALU_MFMA_BUSY_CYCLES (summed over all SIMDs, in cycles) and
    GRBM_GUI_ACTIVE (GPU busy cycles, summed over the 8 XCDs), over the
    product's dispatches after the reference copy: busy / (simds x
    GRBM_GUI_ACTIVE / 8) -- which counts the gaps between dispatches under
    the profiler as busy time -- and, given a kernel-trace run of the same
    command, busy / (simds x kernel duration x clock), over the kernel's own
    duration at the 2.4 GHz peak clock (SQ_VALU_MFMA_BUSY_CYCLES counts the
    instructions' issue cycles, the same for every launch, so the steady
    warm-up launches' duration gives the timed steps' share).""" 
    path = sorted(glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True))
    if not path:
        raise SystemExit(f"no counter_collection.csv under {pmc_dir}")
    per = OrderedDict()
    for r in _rows(path[0]):
        d = int(r["Dispatch_Id"])
        per.setdefault(d, {"name": r["Kernel_Name"], "grid": r.get("Grid_Size")})
        per[d][r["Counter_Name"]] = per[d].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    rows = [v for _, v in sorted(per.items())]
    last_copy = max(i for i, v in enumerate(rows) if "copyBuffer" in v["name"] or "copy_kernel" in v["name"])
    mine = [v for v in rows[last_copy + 1:] if "nnjit" in v["name"]]
    tot = {}
    for v in mine:
        for k, x in v.items():
            if k not in ("name", "grid"):
                tot[k] = tot.get(k, 0.0) + x
    reps = meta["reps"]
    busy = tot.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / reps
    gui = tot.get("GRBM_GUI_ACTIVE", 0.0) / reps
    out = {k: round(x / reps, 1) for k, x in sorted(tot.items())}
    out["mfma_busy_fraction"] = round(busy / (simds * gui / 8.0), 4) if gui > 0 else None
    out["kernels"] = sorted({_short(v["name"]) for v in mine})
    if trace_dir:
        dur, steady, names = kernel_duration_us(trace_dir)
        if dur:
            out["trace_kernels"] = names
            out["kernel_duration_us_after_copy"] = round(dur, 2)
            out["mfma_busy_of_kernel_duration_after_copy"] = round(busy / (simds * dur * 1e-6 * clock_ghz * 1e9), 4)
        if steady:
            out["kernel_duration_us_steady"] = round(steady, 2)
            out["mfma_busy_of_kernel_duration"] = round(busy / (simds * steady * 1e-6 * clock_ghz * 1e9), 4)
    return out


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("out_dir", nargs="?")
    ap.add_argument("--last", type=int, default=0, help="only the last N dispatches in the per-grid table")
    ap.add_argument("--top", type=int, default=12)
    ap.add_argument("--traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="counter runs of bench.py --profile-op: record HBM bytes per launch")
    ap.add_argument("--meta", help="file holding the metadata line bench.py --profile-op printed")
    ap.add_argument("--db", help="traffic database (JSON) to add the entry to")
    ap.add_argument("--trace", metavar="KT_DIR",
                    help="with --mfma: a kernel-trace run of the same product (--profile-op), whose mean kernel "
                         "duration normalises the busy cycles")
    ap.add_argument("--mfma", metavar="PMC_DIR",
                    help="counter run of bench.py --profile-op with SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE: "
                         "matrix-core busy fraction of the product")
    a = ap.parse_args(argv)
    if a.mfma:
        import json
        with open(a.meta) as f:
            meta = next(json.loads(l) for l in f if l.startswith("{"))
        print(json.dumps(mfma_busy(a.mfma, meta, trace_dir=a.trace), indent=1))
        return 0
    if a.traffic:
        import json
        with open(a.meta) as f:
            meta = next(json.loads(l) for l in f if l.startswith("{"))
        entry = traffic(a.traffic[0], a.traffic[1], meta)
        key = f"{meta['workload']}|{meta['op']}|{meta['config']}|{meta['split']}"
        print(key, json.dumps(entry, indent=1))
        if a.db:
            db = {}
            if os.path.exists(a.db):
                with open(a.db) as f:
                    db = json.load(f)
            db[key] = entry
            with open(a.db, "w") as f:
                json.dump(db, f, indent=1, sort_keys=True)
                f.write("\n")
        return 0
    print(summarize(a.out_dir, a.last, a.top))
    return 0


if __name__ == "__main__":
    sys.exit(main())
