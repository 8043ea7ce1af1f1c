"""Offline primitive microbenchmark (the paper's web-guided space reduction,
Sec. 5.1 and Fig. 9, on gfx950).

On one large MatMul (default 4096^3) every group of compiled configurations
that differ in exactly one primitive -- double buffering (LDS stages),
register prefetch depth, K-slab depth, matrix-core instruction shape, vector
(16-byte) or element loads -- is timed, one variable at a time.  For each
primitive and setting the report gives how often that setting was the
fastest of its group and its geometric-mean slowdown against the group's
best.  A setting that wins (almost) everywhere is a "consistent" primitive:
the paper fixes those offline and searches only the rest per shape; here the
report is the evidence for the fixed template choices of the kernel families.

    python -m paper_2309_08978_amd.microbench [--dtype f32|f16] [--size 4096] [--reps 3]

Needs a GPU; calls the library through the C-ABI with forced configurations.
"""
from __future__ import annotations

import argparse
import json
import math
import time
from collections import defaultdict

import paper_2309_08978_amd as nj

PRIMITIVES = {
    "stages": "LDS stages (double buffering)",
    "prefetch": "slabs in flight (register prefetch depth)",
    "Kt": "K slab depth",
    "mfma": "matrix-core instruction shape",
    "vec": "bytes per global load (vectorize)",
}
DERIVED = {"id", "name", "lds", "est_regs", "threads"}


def groups_for(cfgs, prim):
    """Configurations (split 1) keyed by every field but `prim` and the
    derived ones; groups with at least two settings of `prim`."""
    g = defaultdict(list)
    for c in cfgs:
        if c["split"] != 1:
            continue
        key = tuple(sorted((k, v) for k, v in c.items() if k not in DERIVED and k != prim))
        g[key].append(c)
    return [v for v in g.values() if len({c[prim] for c in v}) >= 2]


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--dtype", default="f32", choices=["f32", "f16"])
    ap.add_argument("--size", type=int, default=4096)
    ap.add_argument("--reps", type=int, default=3, help="timed launches per configuration (after one warm-up)")
    ap.add_argument("--json", action="store_true", help="print one JSON line instead of the table")
    a = ap.parse_args(argv)

    import torch
    nj.load()
    n = a.size
    tdt = torch.float16 if a.dtype == "f16" else torch.float32
    A = torch.randn(n, n, device="cuda:0").to(tdt)
    B = torch.randn(n, n, device="cuda:0").to(tdt)
    C = torch.empty(n, n, device="cuda:0")
    fam = "gemm_" + a.dtype
    cfgs = [c for c in nj.configs() if c["family"] == fam]
    t0 = time.perf_counter()
    cache = {}

    def timed(c):
        if c["id"] in cache:
            return cache[c["id"]]
        nj.matmul(A, B, C, cfg=c["id"])               # warm-up
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(a.reps):
            nj.matmul(A, B, C, cfg=c["id"])
        e1.record()
        torch.cuda.synchronize()
        cache[c["id"]] = e0.elapsed_time(e1) * 1e3 / a.reps
        return cache[c["id"]]

    report = {}
    for prim, label in PRIMITIVES.items():
        wins, ratios, ngroups = defaultdict(int), defaultdict(list), 0
        for grp in groups_for(cfgs, prim):
            ts = {c["id"]: timed(c) for c in grp}
            best = min(ts.values())
            ngroups += 1
            fastest = min(grp, key=lambda c: ts[c["id"]])
            wins[fastest[prim]] += 1
            for c in grp:
                ratios[c[prim]].append(ts[c["id"]] / best)
        report[prim] = {"label": label, "groups": ngroups,
                        "settings": {str(v): {"wins": wins[v], "groups": len(ratios[v]),
                                              "geomean_slowdown": round(math.exp(sum(map(math.log, r)) / len(r)), 3)}
                                     for v, r in sorted(ratios.items())}}
    elapsed = time.perf_counter() - t0
    if a.json:
        print(json.dumps({"dtype": a.dtype, "size": n, "timed_configs": len(cache), "seconds": round(elapsed, 2),
                          "primitives": report}))
        return 0
    print(f"{fam} on {n}^3: {len(cache)} configurations timed in {elapsed:.2f} s")
    for prim, r in report.items():
        print(f"  {r['label']} ({r['groups']} groups differing only in it):")
        for v, x in r["settings"].items():
            print(f"    {prim}={v:>4}: fastest in {x['wins']:3d} of {x['groups']:3d} groups, "
                  f"geomean slowdown vs the group's best {x['geomean_slowdown']:.3f}")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
