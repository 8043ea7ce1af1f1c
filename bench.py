"""Benchmark of the lite-space tuned MatMul / BatchMatMul / GEMV path on one
MI355X.

A step is one pass over every product of a workload (default: the BART-base
encoder layer at seq 128, fp32: fused QKV, out-proj, FFN-up, FFN-down
linears and the two 12-head attention BatchMatMuls), each product through
the C-ABI on its tuned configuration.  Before timing, every shape is tuned
just in time (``nnjit_tune``), and the tune wall time is reported per shape.
The timed steps replay a HIP graph captured from the eager ABI calls (the
product is launch-bound at these sizes); the eager step time is reported
beside it.  Inputs are resident in HBM when timing starts.

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
COLD_BYTES = 1 << 30  # rotate >= 1 GiB of weights for bandwidth-bound workloads (MALL is 256 MB)


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
    """Device operands of one product and the call that runs it."""

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
        # the weight operand is rotated over `copies` replicas (cold HBM protocol)
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
    """The oracle (CPU, fp64) on the same workload: whole steps, repeated
    until about `budget_s` seconds of CPU work have run (at least one step)."""
    import oracle
    ops = workloads.workload(name)
    inputs = []
    flops = 0
    for i, op in enumerate(ops):
        if op.flops > 5e9:
            continue  # larger products are left out of the CPU sample
        inputs.append((op, workloads.op_inputs(name, i)))
        flops += op.flops
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
    n_ops = len(inputs)
    return {"value": flops * steps / dt / 1e9, "unit": "GFLOP/s", "cores": oracle.max_threads(), "kind": "oracle",
            "sample": f"{steps} full step(s) of {n_ops}/{len(ops)} products ({flops / 1e9:.3f} GFLOP each step), "
                      f"fp64 {'dequantise-and-sum loop' if ops[0].dtype == 'q4' else 'triple loop'}, {dt:.1f} s"}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="bart_base_layer_seq128_f32", choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--kernel-reps", type=int, default=50, help="launches per event-timed burst per product")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager", action="store_true", help="time eager ABI calls instead of the graph replay")
    ap.add_argument("--tuned-cache", default=None,
                    help="kernel database file: loaded before tuning if it exists, written after")
    ap.add_argument("--copy-ref-mb", type=int, default=0,
                    help="first run a plain device copy of this many MiB (reference for HBM counter scaling)")
    ap.add_argument("--profile-op", default=None,
                    help="counter-collection mode: tune, run the reference copy, then launch only this product "
                         "--kernel-reps times and print one metadata line")
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

    weight_bytes = sum(op.weight_bytes for op in ops)
    cold = all(op.kind in ("gemv", "gemv_q4") for op in ops)
    copies = max(1, math.ceil(COLD_BYTES / weight_bytes)) if cold else 1
    runs = [OpRun(name, i, copies) for i in range(len(ops))]
    torch.cuda.synchronize()

    if args.tuned_cache and os.path.exists(args.tuned_cache):
        loaded = nj.check(nj.nnjit_cache_load(args.tuned_cache))
        log(f"[bench] loaded {loaded} tuned shapes from {args.tuned_cache}")

    # just-in-time tuning of every shape
    tunes = []
    for r in runs:
        op = r.op
        t0 = time.perf_counter()
        cfg = nj.check(_tune(op))
        host_ms = (time.perf_counter() - t0) * 1e3
        st = nj.nnjit_last_tune_stats()
        info = nj.nnjit_config_info(cfg)
        tunes.append({"op": op.name, "cfg": cfg, "tune_ms": round(st["wall_ms"], 1), "host_ms": round(host_ms, 1),
                      "lite": st["n_lite"], "timed": st["n_timed"], "aborted": st["n_aborted"],
                      "best_us": round(st["best_us"], 3), "default_us": round(st["default_us"], 3),
                      "config": info.split(" ", 2)[2].split(" threads=")[0]})
        log(f"[bench] tuned {op.name}: {tunes[-1]}")
    if args.tuned_cache:
        nj.check(nj.nnjit_cache_save(args.tuned_cache))

    if args.copy_ref_mb > 0:
        src = torch.ones(args.copy_ref_mb << 18, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if args.profile_op is not None:
        # counter-collection mode: after the reference copy, only this
        # product runs (kernel_reps launches, rotating weight replicas)
        idx = next(i for i, r in enumerate(runs) if r.op.name == args.profile_op)
        r = runs[idx]
        for i in range(args.kernel_reps):
            r.call(i)
        torch.cuda.synchronize()
        t = tunes[idx]
        print(json.dumps({"workload": name, "op": r.op.name, "config": t["config"].split()[0].split("=", 1)[1],
                          "split": int(t["config"].rsplit("split=", 1)[1]), "reps": args.kernel_reps,
                          "copy_ref_mb": args.copy_ref_mb, "algorithmic_bytes": r.op.bytes,
                          "digest": nj.kernel_digest()}), flush=True)
        return 0

    def step(k=0):
        for r in runs:
            r.call(k)

    # eager warm-up (allocates split-K scratch) and eager timing
    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    n_eager = max(1, min(args.steps, 200))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for k in range(n_eager):
        step(k)
    e1.record()
    torch.cuda.synchronize()
    eager_ms = e0.elapsed_time(e1) / n_eager

    # graph of `per_graph` consecutive steps: at least one per weight replica,
    # and enough steps (up to ~0.5 ms of work) that the per-replay launch
    # cost of the graph is amortised
    per_graph = copies
    if eager_ms < 0.5:
        per_graph = max(copies, min(64, math.ceil(0.5 / max(eager_ms, 1e-3))))
    graph = rest = None
    if not args.eager:
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

        per_graph = min(per_graph, args.steps)
        graph = capture(per_graph)
        if args.steps % per_graph:
            rest = capture(args.steps % per_graph)   # the timed region runs exactly --steps steps
        for _ in range(max(1, args.warmup // per_graph)):
            graph.replay()
        if rest is not None:
            rest.replay()
        torch.cuda.synchronize()

    # timed region
    replays = args.steps // per_graph if graph is not None else args.steps
    nsteps = args.steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    if graph is not None:
        for _ in range(replays):
            graph.replay()
        if rest is not None:
            rest.replay()
    else:
        for k in range(args.steps):
            step(k)
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = e0.elapsed_time(e1) / nsteps
    total_flops = sum(op.flops for op in ops)
    total_bytes = sum(op.bytes for op in ops)

    # per-product kernel durations: a captured burst of back-to-back launches
    # (cold replicas for bandwidth-bound workloads) replayed between HIP
    # events on the replaying stream, per-launch median over 3 replays; the
    # same burst issued eagerly and the host-visible latency of one
    # event-bracketed launch are kept beside it
    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    per_op = []
    for r in runs:
        # graph of kernel_reps back-to-back launches: no host work between them
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            r.call(0, side)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        gb = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gb, stream=side):
            for i in range(args.kernel_reps):
                r.call(i, side)
        gb.replay()
        bursts, ebursts = [], []
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            gb.replay()
            b.record(stream)
            bursts.append((a, b))
        for _ in range(3):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for i in range(args.kernel_reps):
                r.call(i)
            b.record(stream)
            ebursts.append((a, b))
        singles = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(10)]
        for i, (a, b) in enumerate(singles):
            a.record(stream)
            r.call(i)
            b.record(stream)
        torch.cuda.synchronize()
        del gb
        us = statistics.median(a.elapsed_time(b) * 1e3 / args.kernel_reps for a, b in bursts)
        eus = statistics.median(a.elapsed_time(b) * 1e3 / args.kernel_reps for a, b in ebursts)
        single = statistics.median(a.elapsed_time(b) * 1e3 for a, b in singles)
        op = r.op
        rl = roofline_of(op, us)
        per_op.append({"op": op.name, "shape_MKN": [op.M, op.K, op.N], "batch": op.batch, "dtype": op.dtype,
                       "us_per_launch": round(us, 3), "us_per_launch_eager": round(eus, 3),
                       "us_single_launch": round(single, 3),
                       "gflops": round(op.flops / us / 1e3, 1),
                       "pct_mfma_peak": (round(100 * op.flops / us / 1e6 / PEAK_TFLOPS[op.dtype], 2)
                                         if op.dtype in PEAK_TFLOPS else None),
                       "gbs": round(op.bytes / us / 1e3, 1), "pct_hbm": round(100 * op.bytes / us / 1e3 / PEAK_HBM_GBS, 2),
                       "bound": rl["bound"], "pct_roofline": round(100 * rl["frac"], 2)})
    dom = max(range(len(runs)), key=lambda i: per_op[i]["us_per_launch"])
    rl = roofline_of(runs[dom].op, per_op[dom]["us_per_launch"])
    cfg_fields = dict(kv.split("=", 1) for kv in nj.nnjit_config_info(tunes[dom]["cfg"]).split() if "=" in kv)
    dop = runs[dom].op
    if cfg_fields["family"].startswith("gemm"):
        wgs = -(-dop.M // int(cfg_fields["Mt"])) * -(-dop.N // int(cfg_fields["Nt"])) * int(cfg_fields["split"])
    elif dop.dtype == "q4":
        wgs = -(-dop.N // int(cfg_fields["rows_per_wg"]))
    else:
        wgs = -(-dop.N // int(cfg_fields["cols"])) * int(cfg_fields["split"])
    rl["traffic"] = measured_traffic(args.traffic_db, name, dop.name, tunes[dom]["config"])
    rl.update({"kernel_op": per_op[dom]["op"], "kernel_config": tunes[dom]["config"],
               "kernel_grid_wgs": wgs, "kernel_grid_z": dop.batch,
               "per_launch": ("flops" if rl["bound"] == "mfma" else "bytes"),
               "algorithmic": runs[dom].op.flops if rl["bound"] == "mfma" else runs[dom].op.bytes,
               "avg_launch_us": per_op[dom]["us_per_launch"]})

    value = total_flops / (ms_per_step * 1e-3) / 1e9
    dt = ops[0].dtype
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GFLOP/s", "n_gpus": 1, "steps": nsteps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dt, "data": "synthetic",
        "config": {"workload": name, "products": [[op.name, op.batch, op.M, op.K, op.N] for op in ops],
                   "timing": "graph replay" if graph is not None else "eager ABI calls",
                   "weight_replicas": copies, "steps_per_graph": per_graph if graph is not None else None},
        "pct_mfma_peak": round(100 * value / 1e3 / PEAK_TFLOPS[dt], 2) if dt in PEAK_TFLOPS else None,
        "gbs": round(total_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "eager_ms_per_step": round(eager_ms, 5),
        "wall_s": round(wall, 4),
        "tune": tunes,
        "tune_ms_max": max(t["tune_ms"] for t in tunes),
        "per_op": per_op,
        "roofline": rl,
        "device": torch.cuda.get_device_name(0),
    }
    if args.online_steps > 0:
        out["online"] = online_curve(runs, args.online_steps)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(name, args.cpu_budget)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
