"""Offline primitive microbenchmark (the paper's web-guided space reduction,
Sec. 5.1 and Fig. 9, on gfx950).

On MatMuls of fixed sizes (default 4096^3 and 64x768x768) every group of
compiled configurations that differ in exactly one primitive is timed, one
variable at a time: staging of the slabs (through registers, or direct
global->LDS copies), the A slab's LDS layout (XOR swizzle, padding, plain),
a fully unrolled or rolled K-step loop, double buffering (LDS stages),
register prefetch depth, K-slab depth, matrix-core instruction shape, and
vector (16-byte) or element loads.  For each primitive and setting the
report gives how often that setting was the fastest of its group and its
geometric-mean slowdown against the group's best.

A setting that is the fastest in every group of its primitive at every size,
with every other setting at least 5% slower on geometric mean, is a
"consistent" primitive: the paper fixes those offline and searches only the
rest per shape.  ``--save FILE`` stores the measurement; ``--write-table``
turns a stored measurement into ``csrc/consistent.inc``, the table of fixed
settings that the lite-space builder applies (a configuration with another
setting of a consistent primitive never enters a lite space when a twin of
it with the fixed setting is compiled).

    python -m paper_2309_08978_amd.microbench [--dtype f32|f16|all] [--reps 3] [--save FILE] [--json]
    python -m paper_2309_08978_amd.microbench --write-table [FILE]

Timing needs a GPU (the library through its C-ABI with forced
configurations); --write-table is host-only.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import time
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
MEASUREMENT = os.path.join(HERE, "microbench_gfx950.json")
TABLE = os.path.join(HERE, "csrc", "consistent.inc")

PRIMITIVES = {
    "direct": "slab staging: registers (0) or direct global->LDS copies (1)",
    "layout": "A slab layout in LDS (XOR swizzle / padding / plain)",
    "unroll": "K steps of a slab (fully unrolled / rolled loop)",
    "stages": "LDS stages (double buffering)",
    "prefetch": "slabs in flight (register prefetch depth)",
    "Kt": "K slab depth",
    "mfma": "matrix-core instruction shape",
    "vec": "bytes per global load (vectorize)",
}
DERIVED = {"id", "name", "lds", "est_regs", "threads"}
# configuration fields that define a "direct" group: the tile hierarchy, the
# instruction shape and the load width (the kernels of the two staging kinds
# differ in their other fields by construction)
DIRECT_KEY = ("family", "mfma", "Mt", "Nt", "Kt", "waves", "vec", "split")
SIZES = [(4096, 4096, 4096), (64, 768, 768)]   # (M, N, K)
MARGIN = 1.05
FAMILY_ENUM = {"gemm_f32": "FAM_GEMM_F32", "gemm_f16": "FAM_GEMM_F16"}
PRIM_ENUM = {"direct": "PRIM_DIRECT", "layout": "PRIM_LAYOUT", "unroll": "PRIM_UNROLL", "stages": "PRIM_STAGES",
             "prefetch": "PRIM_PREFETCH", "Kt": "PRIM_KT", "mfma": "PRIM_MFMA", "vec": "PRIM_VEC"}


def setting_value(prim: str, v) -> int:
    """The integer a setting is stored as in the C table (Variant fields)."""
    if prim == "layout":
        return {"swz": 0, "pad": 1, "plain": 2}[v]
    if prim == "unroll":
        return {"full": 0, "rolled": 1}[v]
    if prim == "mfma":
        return int(str(v).split("x")[0])
    return int(v)


def groups_for(cfgs, prim):
    """Groups of configurations (split 1) that differ only in `prim`, each a
    dict setting -> [configurations]; groups with at least two settings."""
    g = defaultdict(lambda: defaultdict(list))
    for c in cfgs:
        if c["split"] != 1:
            continue
        if prim == "direct":
            key = tuple(c[k] for k in DIRECT_KEY)
        else:
            key = tuple(sorted((k, v) for k, v in c.items() if k not in DERIVED and k != prim))
        g[key][c[prim]].append(c)
    return [dict(v) for v in g.values() if len(v) >= 2]


def group_key(c, prim):
    """The group a configuration belongs to for `prim` (see groups_for)."""
    if prim == "direct":
        return tuple(c[k] for k in DIRECT_KEY[:-1])
    return tuple(sorted((k, v) for k, v in c.items() if k not in DERIVED and k not in (prim, "split")))


def excluded_by(c, fixed, cfgs):
    """The fixed settings (family, primitive, setting, kinds) that exclude
    configuration c from lite spaces: c has another setting of the
    primitive, and a twin of c (same group) with the fixed setting exists --
    the rule the lite-space builder applies."""
    out = []
    for fam, prim, v, kinds in fixed:
        if c["family"] != fam or c["direct"] not in kinds or str(c[prim]) == str(v):
            continue
        if any(str(u[prim]) == str(v) and group_key(u, prim) == group_key(c, prim)
               for u in cfgs if u["family"] == fam and u["split"] == 1):
            out.append((prim, v))
    return out


def measure(dtype: str, size, reps: int):
    """One size, one dtype: the per-primitive report and the configurations
    (scope) each primitive's groups covered."""
    import torch
    import paper_2309_08978_amd as nj
    nj.load()
    M, N, K = size
    tdt = torch.float16 if dtype == "f16" else torch.float32
    A = torch.randn(M, K, device="cuda:0").to(tdt)
    B = torch.randn(K, N, device="cuda:0").to(tdt)
    C = torch.empty(M, N, device="cuda:0")
    fam = "gemm_" + dtype
    cfgs = [c for c in nj.configs() if c["family"] == fam]
    cache = {}

    def timed(c):
        if c["id"] in cache:
            return cache[c["id"]]
        nj.matmul(A, B, C, cfg=c["id"])               # warm-up
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            nj.matmul(A, B, C, cfg=c["id"])
        e1.record()
        torch.cuda.synchronize()
        cache[c["id"]] = e0.elapsed_time(e1) * 1e3 / reps
        return cache[c["id"]]

    t0 = time.perf_counter()
    report = {}
    for prim, label in PRIMITIVES.items():
        wins, ratios, ngroups, kinds = defaultdict(int), defaultdict(list), 0, set()
        for grp in groups_for(cfgs, prim):
            best_of = {v: min(timed(c) for c in cs) for v, cs in grp.items()}
            best = min(best_of.values())
            ngroups += 1
            wins[min(best_of, key=best_of.get)] += 1
            for v, t in best_of.items():
                ratios[v].append(t / best)
            kinds |= {c["direct"] for cs in grp.values() for c in cs}
        report[prim] = {"label": label, "groups": ngroups, "staging_kinds": sorted(kinds),
                        "settings": {str(v): {"wins": wins[v], "groups": len(r),
                                              "geomean_slowdown": round(math.exp(sum(map(math.log, r)) / len(r)), 3)}
                                     for v, r in sorted(ratios.items(), key=lambda kv: str(kv[0]))}}
    return {"dtype": dtype, "size": list(size), "timed_configs": len(cache),
            "seconds": round(time.perf_counter() - t0, 3), "primitives": report}


def consistent_settings(runs):
    """[(family, primitive, setting, staging kinds)] of the consistent
    primitives of a stored measurement (see the module docstring)."""
    out = []
    for dtype in sorted({r["dtype"] for r in runs}):
        rs = [r for r in runs if r["dtype"] == dtype]
        for prim in PRIMITIVES:
            with_groups = [r["primitives"][prim] for r in rs if r["primitives"][prim]["groups"] > 0]
            if not with_groups:
                continue
            cands = None
            for p in with_groups:
                ok = set()
                for v, x in p["settings"].items():
                    others = [y["geomean_slowdown"] for w, y in p["settings"].items() if w != v]
                    if x["groups"] == p["groups"] and x["wins"] == p["groups"] and others and min(others) >= MARGIN:
                        ok.add(v)
                cands = ok if cands is None else cands & ok
            for v in sorted(cands or ()):
                kinds = sorted(set().union(*(set(p["staging_kinds"]) for p in with_groups)))
                out.append(("gemm_" + dtype, prim, v, kinds))
    return out


def table_text(runs) -> str:
    lines = ["// Consistent primitives of the GEMM families (Sec. 5.1): settings fixed offline.",
             "// Generated by `python -m paper_2309_08978_amd.microbench --write-table` from",
             "// paper_2309_08978_amd/microbench_gfx950.json; do not edit by hand.",
             "// {family, primitive, setting, applies to register-staged, applies to direct-copy}"]
    for fam, prim, v, kinds in consistent_settings(runs):
        lines.append(f"{{{FAMILY_ENUM[fam]}, {PRIM_ENUM[prim]}, {setting_value(prim, v)}, "
                     f"{1 if 0 in kinds else 0}, {1 if 1 in kinds else 0}}},  // {prim}={v}")
    return "\n".join(lines) + "\n"


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--dtype", default="all", choices=["f32", "f16", "all"])
    ap.add_argument("--reps", type=int, default=3, help="timed launches per configuration (after one warm-up)")
    ap.add_argument("--json", action="store_true", help="print one JSON line instead of the table")
    ap.add_argument("--save", metavar="FILE", help="store the measurement (JSON)")
    ap.add_argument("--write-table", nargs="?", const=MEASUREMENT, metavar="FILE",
                    help="write csrc/consistent.inc from a stored measurement (default: the committed one)")
    a = ap.parse_args(argv)
    if a.write_table:
        with open(a.write_table) as f:
            runs = json.load(f)["runs"]
        with open(TABLE, "w") as f:
            f.write(table_text(runs))
        print(open(TABLE).read(), end="")
        return 0

    dtypes = ["f32", "f16"] if a.dtype == "all" else [a.dtype]
    runs = [measure(dt, size, a.reps) for dt in dtypes for size in SIZES]
    if a.save:
        with open(a.save, "w") as f:
            json.dump({"device": "gfx950", "margin": MARGIN, "runs": runs}, f, indent=1)
            f.write("\n")
    if a.json:
        print(json.dumps({"runs": runs, "consistent": consistent_settings(runs)}))
        return 0
    for r in runs:
        M, N, K = r["size"]
        print(f"gemm_{r['dtype']} on {M}x{N}x{K}: {r['timed_configs']} configurations timed in {r['seconds']:.2f} s")
        for prim, p in r["primitives"].items():
            print(f"  {p['label']} ({p['groups']} groups differing only in it):")
            for v, x in p["settings"].items():
                print(f"    {prim}={v:>6}: fastest in {x['wins']:3d} of {x['groups']:3d} groups, "
                      f"geomean slowdown vs the group's best {x['geomean_slowdown']:.3f}")
    print("consistent (fixed offline):")
    for fam, prim, v, kinds in consistent_settings(runs):
        print(f"  {fam}: {prim}={v} (staging kinds {kinds})")
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
