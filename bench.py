"""Benchmark of the lite-space tuned MatMul / BatchMatMul / GEMV path on one
MI355X.

A step is one pass over every product of a workload, each product through
the C-ABI on its tuned configuration.  The default workload is the largest
one that fits one GPU: the Llama-2-7B prefill of 512 tokens in fp32 (the
QKV, out-proj, gate/up, down and LM-head linears and the two 32-head causal
attention BatchMatMuls).  Before timing, every shape is tuned just in time
(``nnjit_tune``) and the tune wall time is reported per shape.  The timed
steps replay a HIP graph captured from the eager ABI calls; the eager step
time is reported beside it.  Inputs are resident in HBM when timing starts.

Besides the headline workload, every other workload (the single
64x768x768 product, the BART-base and T5-large layers, the Llama-2-7B
decode GEMVs with fp32, fp16 and 4-bit weights, the fp16 prefill and the
paper's Table 3 kernels) is tuned and measured per product in the same run
and reported under ``workloads``; ``--only`` skips them.

Prints ONE JSON line.  ``--gpus N`` with N > 1 is refused: the library runs
on one GPU (products are not sharded across devices).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2309_08978_amd as nj  # noqa: E402
import workloads  # noqa: E402

METRIC = "GFLOP/s (%MFMA peak) per GEMM shape; GB/s (%HBM) for GEMV; tune time"
PEAK_TFLOPS = {"f32": 157.3, "f16": 2516.6}  # dense MFMA peaks of MI355X
PEAK_HBM_GBS = 8000.0
RIDGE = {dt: PEAK_TFLOPS[dt] * 1e12 / (PEAK_HBM_GBS * 1e9) for dt in PEAK_TFLOPS}
COLD_BYTES = 1 << 30  # rotate >= 1 GiB of weights per product for bandwidth-bound workloads (MALL is 256 MB)
HEADLINE = "llama2_7b_prefill512_f32"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _kind(op):
    return {"gemm": nj.NNJIT_KIND_GEMM, "batched": nj.NNJIT_KIND_BATCHED, "gemv": nj.NNJIT_KIND_GEMV,
            "gemv_q4": nj.NNJIT_KIND_GEMV_Q4}[op.kind]


def _dt(op):
    return nj.NNJIT_F16 if op.dtype in ("f16", "q4") else nj.NNJIT_F32


def _key(op):
    """(kind, dtype, batch, M, N, K) of a product in the tuned cache (a 4-bit
    GEMV is keyed by its group size in the batch position)."""
    return (_kind(op), _dt(op), op.group if op.dtype == "q4" else op.batch, op.M, op.N, op.K)


def _tune(op):
    if op.dtype == "q4":
        return nj.nnjit_tune_gemv_q4(op.N, op.K, op.group)
    if op.batch > 1:
        return nj.nnjit_tune_batched(op.batch, op.M, op.N, op.K, _dt(op))
    return nj.nnjit_tune(op.M, op.N, op.K, _dt(op))


class OpRun:
    """Device operands of one product and the call that runs it.  The weight
    operand has `copies` replicas that consecutive calls rotate over."""

    def __init__(self, name, index, copies):
        import torch
        self.op = op = workloads.workload(name)[index]
        ins = workloads.op_inputs(name, index)
        self.A = torch.from_numpy(ins[0]).to("cuda:0")
        if op.dtype == "q4":
            # the weight operand is (code words, scales)
            w0 = (torch.from_numpy(ins[1].view(np.int32)).to("cuda:0"), torch.from_numpy(ins[2]).to("cuda:0"))
            clone = lambda w: (w[0].clone(), w[1].clone())
        else:
            w0 = torch.from_numpy(ins[1]).to("cuda:0")
            clone = lambda w: w.clone()
        self.Bs = [w0] + [clone(w0) for _ in range(copies - 1)]
        shape = (op.batch, op.M, op.N) if op.batch > 1 else ((op.N,) if op.dtype == "q4" else (op.M, op.N))
        self.C = torch.empty(shape, dtype=torch.float32, device="cuda:0")

    def call(self, copy=0, stream=None):
        import torch
        if stream is None:
            stream = torch.cuda.current_stream()  # the capture stream while a graph is recorded
        op = self.op
        B = self.Bs[copy % len(self.Bs)]
        if op.dtype == "q4":
            Wq, S = B
            rc = nj.nnjit_gemv_q4(op.N, op.K, op.group, self.A, Wq, Wq.shape[1], S, S.shape[1], self.C, stream)
        elif op.batch > 1:
            rc = nj.nnjit_batched_matmul(op.batch, op.M, op.N, op.K, self.A, op.K, op.M * op.K, B, op.N,
                                         op.K * op.N, self.C, op.N, op.M * op.N, _dt(op), stream)
        else:
            rc = nj.nnjit_matmul(op.M, op.N, op.K, self.A, op.K, B, op.N, self.C, op.N, _dt(op), stream)
        if rc != 0:
            raise nj.NnjitError(rc, nj.nnjit_last_error())


def is_cold(ops) -> bool:
    """Bandwidth-bound workloads (GEMVs) are timed on weights streamed from
    HBM, rotating over replicas too large for the 256 MB last-level cache."""
    return all(op.kind in ("gemv", "gemv_q4") for op in ops)


def replicas(op, cold: bool) -> int:
    return max(1, math.ceil(COLD_BYTES / op.weight_bytes)) if cold else 1


def roofline_of(op, us):
    dt = op.dtype
    ai = op.flops / op.bytes
    if dt != "q4" and ai >= RIDGE[dt]:   # the 4-bit GEMV runs no MFMA: HBM is its roofline
        achieved = op.flops / (us * 1e-6) / 1e12
        return {"bound": "mfma", "achieved": achieved, "peak": PEAK_TFLOPS[dt], "unit": "TFLOP/s",
                "frac": achieved / PEAK_TFLOPS[dt], "traffic": None}
    achieved = op.bytes / (us * 1e-6) / 1e9
    return {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS, "traffic": None}


def measured_traffic(db_path, workload, op, config_info):
    """HBM bytes per launch of this product from the counter database, or
    None when it has no entry for the exact configuration or the kernel
    sources changed since the counters were taken."""
    try:
        with open(db_path) as f:
            db = json.load(f)
    except (OSError, ValueError):
        return None
    cfg = config_info.split()[0].split("=", 1)[1]
    split = int(config_info.rsplit("split=", 1)[1])
    e = db.get(f"{workload}|{op}|{cfg}|{split}")
    if not e or e.get("digest") != nj.kernel_digest():
        return None
    return e["hbm_bytes_per_launch"]


def online_curve(runs, nsteps):
    """Per-step time of eager steps from an empty cache with online tuning on:
    each step's calls measure one candidate per untuned shape, so the step
    time falls as registered configurations improve, until every shape is
    tuned (reproduces the paper's speed-up-over-time measurement)."""
    import torch
    nj.nnjit_cache_clear()
    prev = nj.nnjit_set_online(True)
    ms, tuned_at = [], None
    try:
        for k in range(nsteps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for r in runs:
                r.call(k)
            b.record()
            torch.cuda.synchronize()
            ms.append(round(a.elapsed_time(b), 5))
            if tuned_at is None:
                states = [nj.nnjit_online_status(*_key(r.op))["state"] for r in runs]
                if all(st == "tuned" for st in states):
                    tuned_at = k + 1
    finally:
        nj.nnjit_set_online(prev)
    return {"step_ms": ms, "steps_until_all_tuned": tuned_at, "first_ms": ms[0], "last_ms": ms[-1]}


def cpu_baseline(name, budget_s: float):
    """The oracle (CPU, fp64) on whole steps of the same workload -- every
    product of the step -- repeated until about `budget_s` seconds of CPU
    work have run (at least one step)."""
    import oracle
    ops = workloads.workload(name)
    inputs = [(op, workloads.op_inputs(name, i)) for i, op in enumerate(ops)]
    flops = sum(op.flops for op in ops)
    oracle.default()
    t0 = time.perf_counter()
    steps = 0
    while True:
        for op, ins in inputs:
            if op.dtype == "q4":
                oracle.gemv_q4(*ins, op.group, op.N)
            else:
                oracle.matmul(*ins)
        steps += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": flops * steps / dt / 1e9, "unit": "GFLOP/s", "cores": oracle.max_threads(), "kind": "oracle",
            "sample": f"{steps} full step(s) of {len(ops)}/{len(ops)} products ({flops / 1e9:.3f} GFLOP each step), "
                      f"fp64 {'dequantise-and-sum loop' if ops[0].dtype == 'q4' else 'triple loop'}, {dt:.1f} s"}


def tune_all(runs):
    """Just-in-time tuning of every product's shape, with its statistics."""
    tunes = []
    for r in runs:
        op = r.op
        t0 = time.perf_counter()
        cfg = nj.check(_tune(op))
        host_ms = (time.perf_counter() - t0) * 1e3
        st = nj.nnjit_last_tune_stats_ex()
        info = nj.nnjit_config_info(cfg)
        tunes.append({"op": op.name, "cfg": cfg, "tune_ms": round(st["wall_ms"], 1), "host_ms": round(host_ms, 1),
                      "lite": st["n_lite"], "timed": st["n_timed"], "aborted": st["n_aborted"],
                      "best_us": round(st["best_us"], 3), "default_us": round(st["default_us"], 3),
                      "config": info.split(" ", 2)[2].split(" threads=")[0]})
        log(f"[bench] tuned {op.name}: {tunes[-1]}")
    return tunes


def time_steps(runs, steps, warmup, eager_only):
    """Eager and graph-replayed step times.  A graph holds `per_graph`
    consecutive steps -- at least one per weight replica, and for short steps
    enough of them (<= 64, ~0.5 ms of work) that a replay's launch cost is
    amortised -- and a second graph the remainder, so that exactly `steps`
    steps run between the events."""
    import torch

    def step(k=0):
        for r in runs:
            r.call(k)

    for k in range(warmup):    # eager warm-up (allocates split-K scratch)
        step(k)
    torch.cuda.synchronize()
    n_eager = max(1, min(steps, 200))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for k in range(n_eager):
        step(k)
    e1.record()
    torch.cuda.synchronize()
    eager_ms = e0.elapsed_time(e1) / n_eager

    copies = max(len(r.Bs) for r in runs)
    per_graph = copies
    if eager_ms < 0.5:
        per_graph = max(copies, min(64, math.ceil(0.5 / max(eager_ms, 1e-3))))
    graph = rest = None
    if not eager_only:
        side = torch.cuda.Stream()

        def capture(n):
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                for k in range(n):
                    step(k)  # warm-up on the capture stream (its split-K scratch)
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                for k in range(n):
                    step(k)
            return g

        per_graph = min(per_graph, steps)
        graph = capture(per_graph)
        if steps % per_graph:
            rest = capture(steps % per_graph)
        for _ in range(max(1, warmup // per_graph)):
            graph.replay()
        if rest is not None:
            rest.replay()
        torch.cuda.synchronize()

    # timed region
    replays = steps // per_graph if graph is not None else steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    if graph is not None:
        for _ in range(replays):
            graph.replay()
        if rest is not None:
            rest.replay()
    else:
        for k in range(steps):
            step(k)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return {"ms_per_step": e0.elapsed_time(e1) / steps, "eager_ms_per_step": eager_ms, "wall_s": wall,
            "timing": "graph replay" if graph is not None else "eager ABI calls",
            "steps_per_graph": per_graph if graph is not None else None}


def burst_us(fn, reps, stream, side):
    """Device time per call of `fn(i, stream)`: `reps` back-to-back calls
    captured as a graph on `side` and replayed between HIP events on
    `stream`, median of 3 replays; plus the same burst issued eagerly and
    the latency of single event-bracketed calls."""
    import torch
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        fn(0, side)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    gb = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gb, stream=side):
        for i in range(reps):
            fn(i, side)
    gb.replay()
    ev = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    bursts, ebursts = [], []
    for _ in range(3):
        a, b = ev()
        a.record(stream)
        gb.replay()
        b.record(stream)
        bursts.append((a, b))
    for _ in range(3):
        a, b = ev()
        a.record(stream)
        for i in range(reps):
            fn(i, stream)
        b.record(stream)
        ebursts.append((a, b))
    singles = [ev() for _ in range(10)]
    for i, (a, b) in enumerate(singles):
        a.record(stream)
        fn(i, stream)
        b.record(stream)
    torch.cuda.synchronize()
    del gb
    return (statistics.median(a.elapsed_time(b) * 1e3 / reps for a, b in bursts),
            statistics.median(a.elapsed_time(b) * 1e3 / reps for a, b in ebursts),
            statistics.median(a.elapsed_time(b) * 1e3 for a, b in singles))


def stream_ceiling_us(nbytes, copies, reps, stream, side):
    """What one launch can stream: a non-temporal 16-byte-load read (nnjit_stream_read)
    of the same byte count, rotating over the same number of replicas (cold),
    timed like the products; the best of several grid sizes."""
    import torch
    n16 = -(-nbytes // 16) * 16
    bufs = [torch.empty(n16 // 4, dtype=torch.int32, device="cuda:0") for _ in range(copies)]
    for b in bufs:
        b.fill_(1)
    best = None
    for wgs in (256, 512, 1024, 2048, 4096):
        sink = torch.zeros(wgs, dtype=torch.int32, device="cuda:0")

        def fn(i, s, wgs=wgs, sink=sink):
            nj.check(nj.nnjit_stream_read(bufs[i % copies], n16, sink, wgs, s))

        us = burst_us(fn, reps, stream, side)[0]
        best = us if best is None else min(best, us)
    del bufs
    torch.cuda.empty_cache()
    return best


def per_op_times(runs, reps, ceiling):
    import torch
    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    per_op = []
    for r in runs:
        us, eus, single = burst_us(lambda i, s, r=r: r.call(i, s), reps, stream, side)
        op = r.op
        rl = roofline_of(op, us)
        row = {"op": op.name, "shape_MKN": [op.M, op.K, op.N], "batch": op.batch, "dtype": op.dtype,
               "us_per_launch": round(us, 3), "us_per_launch_eager": round(eus, 3),
               "us_single_launch": round(single, 3),
               "gflops": round(op.flops / us / 1e3, 1),
               "pct_mfma_peak": (round(100 * op.flops / us / 1e6 / PEAK_TFLOPS[op.dtype], 2)
                                 if op.dtype in PEAK_TFLOPS else None),
               "gbs": round(op.bytes / us / 1e3, 1), "pct_hbm": round(100 * op.bytes / us / 1e3 / PEAK_HBM_GBS, 2),
               "bound": rl["bound"], "pct_roofline": round(100 * rl["frac"], 2)}
        if ceiling:
            cus = stream_ceiling_us(op.weight_bytes, len(r.Bs), reps, stream, side)
            row["stream_ceiling_gbs"] = round(op.weight_bytes / cus / 1e3, 1)
            row["pct_of_stream_ceiling"] = round(100 * cus / us, 2)
        per_op.append(row)
    return per_op


def dominant_roofline(name, runs, per_op, tunes, traffic_db):
    """roofline object of the product with the most time per step."""
    dom = max(range(len(runs)), key=lambda i: per_op[i]["us_per_launch"])
    dop = runs[dom].op
    rl = roofline_of(dop, per_op[dom]["us_per_launch"])
    cfg_fields = dict(kv.split("=", 1) for kv in nj.nnjit_config_info(tunes[dom]["cfg"]).split() if "=" in kv)
    if cfg_fields["family"].startswith("gemm"):
        wgs = -(-dop.M // int(cfg_fields["Mt"])) * -(-dop.N // int(cfg_fields["Nt"])) * int(cfg_fields["split"])
    elif dop.dtype == "q4":
        wgs = -(-dop.N // int(cfg_fields["rows_per_wg"]))
    else:
        wgs = -(-dop.N // int(cfg_fields["cols"])) * int(cfg_fields["split"])
    rl["traffic"] = measured_traffic(traffic_db, name, dop.name, tunes[dom]["config"])
    rl.update({"kernel_op": per_op[dom]["op"], "kernel_config": tunes[dom]["config"],
               "kernel_grid_wgs": wgs, "kernel_grid_z": dop.batch,
               "per_launch": ("flops" if rl["bound"] == "mfma" else "bytes"),
               "algorithmic": dop.flops if rl["bound"] == "mfma" else dop.bytes,
               "avg_launch_us": per_op[dom]["us_per_launch"]})
    return rl


def measure(name, args, steps, warmup):
    """Tune and time one workload: step times, per-product times, roofline of
    the dominant product.  Frees its device operands before returning."""
    import torch
    ops = workloads.workload(name)
    cold = is_cold(ops)
    runs = [OpRun(name, i, replicas(op, cold)) for i, op in enumerate(ops)]
    torch.cuda.synchronize()
    tunes = tune_all(runs)
    st = time_steps(runs, steps, warmup, args.eager)
    per_op = per_op_times(runs, args.kernel_reps, ceiling=cold and not args.no_stream_ceiling)
    rl = dominant_roofline(name, runs, per_op, tunes, args.traffic_db)
    flops = sum(op.flops for op in ops)
    nbytes = sum(op.bytes for op in ops)
    dt = ops[0].dtype
    out = {"workload": name, "dtype": dt, "value": flops / (st["ms_per_step"] * 1e-3) / 1e9, "unit": "GFLOP/s",
           "pct_mfma_peak": (round(100 * flops / (st["ms_per_step"] * 1e-3) / 1e12 / PEAK_TFLOPS[dt], 2)
                             if dt in PEAK_TFLOPS else None),
           "gbs": round(nbytes / (st["ms_per_step"] * 1e-3) / 1e9, 1), "steps": steps,
           "weight_replicas": max(len(r.Bs) for r in runs), **st,
           "tune": tunes, "tune_ms_max": max(t["tune_ms"] for t in tunes), "per_op": per_op, "roofline": rl,
           "products": [[op.name, op.batch, op.M, op.K, op.N] for op in ops]}
    if args.online_steps > 0 and name == args.workload:
        out["online"] = online_curve(runs, args.online_steps)
    del runs
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def compact(m):
    """The per-product table of a workload measured beside the headline."""
    return {"value": round(m["value"], 1), "unit": m["unit"], "dtype": m["dtype"],
            "ms_per_step": round(m["ms_per_step"], 5), "pct_mfma_peak": m["pct_mfma_peak"], "gbs": m["gbs"],
            "tune_ms_max": m["tune_ms_max"],
            "per_op": [{k: p[k] for k in ("op", "shape_MKN", "batch", "us_per_launch", "gflops", "pct_mfma_peak",
                                          "gbs", "pct_hbm", "bound", "pct_roofline", "stream_ceiling_gbs",
                                          "pct_of_stream_ceiling") if k in p}
                       | {"config": t["config"].split()[0].split("=", 1)[1],
                          "split": int(t["config"].rsplit("split=", 1)[1])}
                       for p, t in zip(m["per_op"], m["tune"])],
            "roofline": {k: m["roofline"][k] for k in ("bound", "achieved", "peak", "unit", "frac", "traffic",
                                                       "kernel_op")}}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=HEADLINE, choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--only", action="store_true", help="measure the headline workload only")
    ap.add_argument("--kernel-reps", type=int, default=50, help="launches per event-timed burst per product")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stream-ceiling", action="store_true",
                    help="skip the streaming-read reference of bandwidth-bound products")
    ap.add_argument("--eager", action="store_true", help="time eager ABI calls instead of the graph replay")
    ap.add_argument("--tuned-cache", default=None,
                    help="kernel database file: loaded before tuning if it exists, written after")
    ap.add_argument("--copy-ref-mb", type=int, default=0,
                    help="first run a plain device copy of this many MiB (reference for HBM counter scaling)")
    ap.add_argument("--profile-op", default=None,
                    help="counter-collection mode: tune, run the reference copy, then launch only this product "
                         "--kernel-reps times and print one metadata line")
    ap.add_argument("--profile-config", default=None,
                    help="with --profile-op: launch this configuration (name or name:split) instead of the tuned one")
    ap.add_argument("--online-steps", type=int, default=0,
                    help="after the measurement, clear the tuned cache and run this many eager steps with online "
                         "just-in-time tuning, reporting each step's time (the gradual speed-up curve)")
    ap.add_argument("--traffic-db", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM traffic per launch (written from rocprofv3 counter runs)")
    args = ap.parse_args(argv)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the library has no multi-GPU path", file=sys.stderr)
        return 2

    import torch
    if not torch.cuda.is_available():
        print("no GPU available", file=sys.stderr)
        return 3
    nj.load()
    torch.cuda.set_device(0)
    name = args.workload
    ops = workloads.workload(name)
    log(f"[bench] workload {name}: {len(ops)} products")

    if args.tuned_cache and os.path.exists(args.tuned_cache):
        loaded = nj.check(nj.nnjit_cache_load(args.tuned_cache))
        log(f"[bench] loaded {loaded} tuned shapes from {args.tuned_cache}")

    if args.profile_op is not None:
        # counter-collection mode: tune, run the reference copy, then launch
        # only this product kernel_reps times (rotating weight replicas)
        cold = is_cold(ops)
        runs = [OpRun(name, i, replicas(op, cold)) for i, op in enumerate(ops)]
        tunes = tune_all(runs)
        if args.tuned_cache:
            nj.check(nj.nnjit_cache_save(args.tuned_cache))
        idx = next(i for i, r in enumerate(runs) if r.op.name == args.profile_op)
        r = runs[idx]
        t = tunes[idx]
        cfg_name, cfg_split = t["config"].split()[0].split("=", 1)[1], int(t["config"].rsplit("split=", 1)[1])
        call = r.call
        if args.profile_config:
            want, _, sp = args.profile_config.partition(":")
            c = next(c for c in nj.configs() if c["name"] == want and (not sp or c["split"] == int(sp)))
            cfg_name, cfg_split = c["name"], c["split"]
            op = r.op

            def call(i, c=c, op=op, r=r):
                B = r.Bs[i % len(r.Bs)]
                if op.batch > 1:
                    nj.check(nj.nnjit_matmul_config(c["id"], op.batch, op.M, op.N, op.K, r.A, op.K, op.M * op.K, B,
                                                    op.N, op.K * op.N, r.C, op.N, op.M * op.N, _dt(op), None))
                else:
                    nj.check(nj.nnjit_matmul_config(c["id"], 1, op.M, op.N, op.K, r.A, op.K, 0, B, op.N, 0, r.C,
                                                    op.N, 0, _dt(op), None))
        # warm-up launches of the product (about half a second), so that the
        # measured ones below run at the clock the timed steps see
        t_end = time.perf_counter() + 0.5
        while time.perf_counter() < t_end:
            for i in range(10):
                call(i)
            torch.cuda.synchronize()
        if args.copy_ref_mb > 0:
            src = torch.ones(args.copy_ref_mb << 18, dtype=torch.float32, device="cuda:0")
            dst = torch.empty_like(src)
            for _ in range(3):
                dst.copy_(src)
            torch.cuda.synchronize()
            del src, dst
        for i in range(args.kernel_reps):
            call(i)
        torch.cuda.synchronize()
        print(json.dumps({"workload": name, "op": r.op.name, "config": cfg_name,
                          "split": cfg_split, "reps": args.kernel_reps,
                          "copy_ref_mb": args.copy_ref_mb, "algorithmic_bytes": r.op.bytes,
                          "digest": nj.kernel_digest()}), flush=True)
        return 0

    head = measure(name, args, args.steps, args.warmup)
    log(f"[bench] {name}: {head['ms_per_step']:.4f} ms/step, {head['value']:.0f} GFLOP/s")
    others = {}
    if not args.only:
        for other in workloads.WORKLOADS:
            if other == name:
                continue
            m = measure(other, args, min(args.steps, 20), min(args.warmup, 3))
            others[other] = compact(m)
            log(f"[bench] {other}: {m['ms_per_step']:.4f} ms/step, {m['value']:.0f} GFLOP/s")
    if args.tuned_cache:
        nj.check(nj.nnjit_cache_save(args.tuned_cache))

    dt = head["dtype"]
    out = {
        "metric": METRIC, "value": round(head["value"], 2), "unit": "GFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(head["ms_per_step"], 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": dt, "data": "synthetic",
        "config": {"workload": name, "products": head["products"], "timing": head["timing"],
                   "weight_replicas": head["weight_replicas"], "steps_per_graph": head["steps_per_graph"]},
        "pct_mfma_peak": head["pct_mfma_peak"],
        "gbs": head["gbs"],
        "eager_ms_per_step": round(head["eager_ms_per_step"], 5),
        "wall_s": round(head["wall_s"], 4),
        "tune": head["tune"],
        "tune_ms_max": head["tune_ms_max"],
        "per_op": head["per_op"],
        "roofline": head["roofline"],
        "device": torch.cuda.get_device_name(0),
    }
    if "online" in head:
        out["online"] = head["online"]
    if others:
        out["workloads"] = others
        out["tune_ms_max_all"] = max([head["tune_ms_max"]] + [o["tune_ms_max"] for o in others.values()])
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(name, args.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
