"""The offline primitive microbenchmark (Sec. 5.1, Fig. 9: one primitive at a
time) on the GPU: a 4096^3 MatMul per family finishes in under a second, every
primitive with groups reports each setting's wins and slowdown, and the
settings the committed table fixes are not contradicted on this device (each
is within the table's margin of the best in this run)."""
import json
import os

import pytest

from paper_2309_08978_amd import microbench as mb

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_microbench_4096_under_a_second(dtype):
    r = mb.measure(dtype, (4096, 4096, 4096), reps=3)
    print(f"{dtype}: {r['timed_configs']} configurations in {r['seconds']:.2f} s", flush=True)
    assert r["seconds"] < 1.0, r["seconds"]
    assert r["timed_configs"] >= 10
    with_groups = [p for p in r["primitives"].values() if p["groups"] > 0]
    assert len(with_groups) >= 3
    for prim, p in r["primitives"].items():
        for v, x in p["settings"].items():
            assert 0 <= x["wins"] <= x["groups"] <= p["groups"]
            assert x["geomean_slowdown"] >= 1.0
        if p["groups"]:
            assert sum(x["wins"] for x in p["settings"].values()) == p["groups"]
    if os.path.exists(mb.MEASUREMENT):
        fixed = mb.consistent_settings(json.load(open(mb.MEASUREMENT))["runs"])
        for fam, prim, v, _ in fixed:
            if fam != "gemm_" + dtype or not r["primitives"][prim]["groups"]:
                continue
            x = r["primitives"][prim]["settings"][v]
            print(f"   fixed {prim}={v}: wins {x['wins']}/{x['groups']}, slowdown {x['geomean_slowdown']}", flush=True)
            assert x["geomean_slowdown"] <= mb.MARGIN, (prim, v, x)
