"""The just-in-time tuner on the GPU (Sec. 3 JIT phase; Sec. 5.2 lite space):
it returns a configuration of the shape's lite space, measured on the
device, within the one-second budget; a second call is a cache hit; a
candidate that fails to launch is skipped; the dispatch then uses the tuned
configuration; and tuned calls replay correctly from a captured HIP graph."""
import os

import numpy as np
import pytest

import oracle
from oracle import accept
import paper_2309_08978_amd as nj
import workloads
from tests.gpu_util import dev, host, kind_of, dtype_code

pytestmark = pytest.mark.gpu

SHAPES = [("matmul_64x768x768_f32", 0)] + [("bart_base_layer_seq128_f32", i) for i in range(6)] + \
         [("llama2_7b_decode_f16", i) for i in (0, 5)] + [("llama2_7b_decode_f32", 4)]


def _tune(op):
    dt = dtype_code(op.dtype)
    if op.batch == 1:
        return nj.nnjit_tune(op.M, op.N, op.K, dt)
    return nj.nnjit_tune_batched(op.batch, op.M, op.N, op.K, dt)


@pytest.mark.parametrize("name,index", SHAPES)
def test_tune_returns_measured_lite_config_within_budget(name, index):
    op = workloads.workload(name)[index]
    dt = dtype_code(op.dtype)
    nj.nnjit_cache_clear()
    cfg = nj.check(_tune(op))
    st = nj.nnjit_last_tune_stats_ex()
    lite, n, n_enum, _ = nj.nnjit_lite_space(kind_of(op.batch, op.M), dt, op.batch, op.M, op.N, op.K)
    print(f"{op.name}: cfg {cfg} {nj.nnjit_config_info(cfg).split()[2]} best {st['best_us']:.2f} us "
          f"(default {st['default_us']:.2f}), lite {st['n_lite']}/{n_enum}, timed {st['n_timed']}, "
          f"aborted {st['n_aborted']}, {st['wall_ms']:.1f} ms", flush=True)
    assert cfg in lite and st["chosen"] == cfg and st["n_lite"] == n
    assert 1 <= st["n_timed"] and st["n_timed"] + st["n_aborted"] + st["n_failed"] <= n
    assert 0 < st["best_us"] <= st["default_us"] * 1.0001 + 1e-9 or st["best_us"] <= st["default_us"] * 1.03
    assert st["wall_ms"] <= 1000.0, st
    # cache hit
    assert _tune(op) == cfg
    st2 = nj.nnjit_last_tune_stats_ex()
    assert st2["cache_hit"] == 1 and st2["wall_ms"] < 5.0
    assert nj.nnjit_cached_config(kind_of(op.batch, op.M), dt, op.batch, op.M, op.N, op.K) == cfg


def test_measured_resources_are_used():
    for c in nj.configs()[::11]:
        r = nj.nnjit_config_resources(c["id"])
        assert r["regs_measured"] == 1 and 0 < r["regs_per_lane"] <= 512
        assert r["wg_per_cu"] >= 1 or c["threads"] > 512


def test_failing_candidate_is_skipped(monkeypatch):
    op = workloads.workload("bart_base_layer_seq128_f32")[1]
    lite, _, _, _ = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K)
    monkeypatch.setenv("NNJIT_FAULT_CONFIG", str(lite[0]))
    nj.nnjit_cache_clear()   # the library reads its environment here
    try:
        cfg = nj.check(nj.nnjit_tune(op.M, op.N, op.K, nj.NNJIT_F32))
        st = nj.nnjit_last_tune_stats_ex()
        assert cfg != lite[0] and cfg in lite and st["n_failed"] >= 1
    finally:
        monkeypatch.delenv("NNJIT_FAULT_CONFIG")
        nj.nnjit_cache_clear()



@pytest.mark.parametrize("graph", ["1", "0"])
def test_graph_and_eager_timing_both_tune(monkeypatch, graph):
    """Candidates are timed as captured graph bursts (default) or, with
    NNJIT_TUNE_GRAPH=0 (the fallback when capture is refused), as eager
    bursts: either way a lite-space configuration is measured, registered,
    and then computes the oracle's exact sums (small integers); a split-K
    GEMV shape exercises the scratch allocated before capture."""
    monkeypatch.setenv("NNJIT_TUNE_GRAPH", graph)
    try:
        _graph_and_eager_timing_both_tune(graph)
    finally:
        monkeypatch.delenv("NNJIT_TUNE_GRAPH")
        nj.nnjit_cache_clear()


def _graph_and_eager_timing_both_tune(graph):
    for name, index in (("bart_base_layer_seq128_f32", 4), ("llama2_7b_decode_f16", 1)):
        op = workloads.workload(name)[index]
        dt = dtype_code(op.dtype)
        nj.nnjit_cache_clear()
        cfg = nj.check(_tune(op))
        st = nj.nnjit_last_tune_stats_ex()
        lite, _, _, _ = nj.nnjit_lite_space(kind_of(op.batch, op.M), dt, op.batch, op.M, op.N, op.K)
        assert cfg in lite and st["n_timed"] >= 1 and st["n_failed"] == 0, st
        A, B = workloads.small_int_operands(8080, op.batch, op.M, op.K, op.N, op.dtype)
        R = oracle.matmul(A, B)
        if op.batch == 1:
            C = nj.matmul(dev(A[0] if A.ndim == 3 else A), dev(B[0] if B.ndim == 3 else B))
        else:
            C = nj.batched_matmul(dev(A), dev(B))
        assert np.array_equal(host(C).reshape(R.shape), R), f"{op.name} graph={graph}"

def test_dispatch_uses_tuned_config_and_matches_oracle():
    name, i = "bart_base_layer_seq128_f32", 3
    op = workloads.workload(name)[i]
    A, B = workloads.op_inputs(name, i)
    nj.nnjit_cache_clear()
    cfg = nj.check(nj.nnjit_tune(op.M, op.N, op.K, nj.NNJIT_F32))
    dA, dB = dev(A), dev(B)
    C_tuned = host(nj.matmul(dA, dB))
    C_forced = host(nj.matmul(dA, dB, cfg=cfg))
    assert np.array_equal(C_tuned, C_forced)
    assert accept.check(C_tuned, oracle.matmul(A, B), A, B, "f32")["ok"]


def test_graph_replay_matches_eager():
    """Tuned calls (split-K included) captured in a graph: every replay,
    with eager work between replays, equals the eager result."""
    import torch
    name = "bart_base_layer_seq128_f32"
    ops = workloads.workload(name)
    ins = [workloads.op_inputs(name, i) for i in range(len(ops))]
    dins = [(dev(A), dev(B)) for A, B in ins]
    for op in ops:
        nj.check(_tune(op))

    def run(stream=None):
        return [nj.matmul(a, b, stream=stream) if a.dim() == 2 else nj.batched_matmul(a, b, stream=stream)
                for a, b in dins]

    eager = [host(c) for c in run()]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        outs = [torch.empty(c.shape, dtype=torch.float32, device="cuda:0") for c in eager]

        def step():
            for (a, b), c in zip(dins, outs):
                (nj.matmul if a.dim() == 2 else nj.batched_matmul)(a, b, c, stream=side)
        step()  # warm-up on the capture stream (allocates its scratch)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        step()
    for rep in range(4):
        for c in outs:
            c.fill_(float("nan"))
        run()  # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        for c, e in zip(outs, eager):
            assert np.array_equal(host(c), e), f"replay {rep}"


def test_capture_refuses_split_k_scratch_growth():
    """A split-K call that would have to grow its stream's scratch while the
    stream is being captured returns NNJIT_EHIP and enqueues nothing; after
    one call outside capture the same call captures and every replay gives
    the oracle's exact sums."""
    import torch
    cfg = next(c for c in nj.configs()
               if c["family"] == "gemm_f32" and c["vec"] == 16 and c["split"] == 4 and not c.get("direct"))
    M, N, K = 64, 192, 512
    A, B = workloads.small_int_operands(4242, 1, M, K, N, "f32")
    R = oracle.matmul(A, B)
    dA, dB = dev(A), dev(B)
    nj.matmul(dA, dB)                     # device state initialised outside any capture
    torch.cuda.synchronize()
    side = torch.cuda.Stream()            # a stream no call has used: no scratch yet
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda:0")
    torch.cuda.synchronize()

    def call():
        return nj.nnjit_matmul_config(cfg["id"], 1, M, N, K, dA, K, 0, dB, N, 0, C, N, 0, nj.NNJIT_F32, side)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        C.fill_(0.0)
        rc = call()
    assert rc == nj.NNJIT_EHIP, rc
    assert "captur" in nj.nnjit_last_error()
    with torch.cuda.stream(side):
        assert call() == nj.NNJIT_OK      # outside capture: the scratch grows
    torch.cuda.synchronize()
    assert np.array_equal(host(C), R)
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=side):
        assert call() == nj.NNJIT_OK
    for rep in range(3):
        C.fill_(float("nan"))
        torch.cuda.synchronize()
        g2.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host(C), R), f"replay {rep}"


def test_kernel_database_roundtrip(tmp_path):
    """Tuned shapes survive a save / clear / load cycle; foreign-device,
    unknown-configuration and malformed lines are skipped."""
    op = workloads.workload("bart_base_layer_seq128_f32")[0]
    nj.nnjit_cache_clear()
    cfg = nj.check(nj.nnjit_tune(op.M, op.N, op.K, nj.NNJIT_F32))
    path = tmp_path / "db.txt"
    assert nj.check(nj.nnjit_cache_save(str(path))) >= 1
    lines = path.read_text().splitlines()
    entry = next(l for l in lines if not l.startswith("#"))
    sig = entry.split()[0]
    with open(path, "a") as f:
        f.write("gfx000:1 " + " ".join(entry.split()[1:]) + "\n")          # another device
        f.write(" ".join([sig] + entry.split()[1:7] + ["no_such_config", "1", "1.0"]) + "\n")
        f.write("garbage line\n")
    nj.nnjit_cache_clear()
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K) == nj.NNJIT_ENOCFG
    assert nj.check(nj.nnjit_cache_load(str(path))) == len([l for l in lines if not l.startswith("#")])
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K) == cfg
    assert nj.check(nj.nnjit_tune(op.M, op.N, op.K, nj.NNJIT_F32)) == cfg
    assert nj.nnjit_last_tune_stats_ex()["cache_hit"] == 1
    assert nj.nnjit_cache_load(str(tmp_path / "missing.txt")) == nj.NNJIT_EINVAL


def test_ranked_candidates_and_database_merge(tmp_path):
    """The database keeps the top-ranked candidates of a shape (registered one
    first) and merging two databases keeps the faster measurement."""
    op = workloads.workload("bart_base_layer_seq128_f32")[1]
    nj.nnjit_cache_clear()
    cfg = nj.check(nj.nnjit_tune(op.M, op.N, op.K, nj.NNJIT_F32))
    ranked = nj.nnjit_cached_ranked(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K)
    st = nj.nnjit_last_tune_stats_ex()
    assert ranked[0][0] == cfg and 1 <= len(ranked) <= 5
    assert len(ranked) == min(5, st["n_timed"])
    assert all(a[1] <= b[1] for a, b in zip(ranked[1:], ranked[2:]))     # the others by time
    assert len({c for c, _ in ranked}) == len(ranked)
    fast = tmp_path / "fast.txt"
    nj.check(nj.nnjit_cache_save(str(fast)))
    line = next(l for l in fast.read_text().splitlines() if not l.startswith("#"))
    f = line.split()
    assert len(f) == 7 + 3 * len(ranked)
    # a second database from an "identical device" with a slower measurement of
    # another configuration: merging keeps the faster one
    other = ranked[1][0] if len(ranked) > 1 else cfg
    slow = tmp_path / "slow.txt"
    oc = nj.configs()[other]
    slow.write_text(" ".join(f[:7] + [oc["name"], str(oc["split"]), f"{ranked[0][1] * 10:.4f}"]) + "\n")
    assert nj.check(nj.nnjit_cache_load(str(slow))) == 1
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K) == cfg
    nj.nnjit_cache_clear()
    assert nj.check(nj.nnjit_cache_load(str(slow))) == 1
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K) == other
    assert nj.check(nj.nnjit_cache_load(str(fast))) == 1                   # faster entry wins
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K) == cfg
    back = nj.nnjit_cached_ranked(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K)
    assert [c for c, _ in back] == [c for c, _ in ranked]          # times are stored to 1e-4 us
    assert all(abs(u - v) <= 1e-4 + 1e-6 * v for (_, u), (_, v) in zip(back, ranked))
    nj.nnjit_cache_clear()


def test_online_tuning_serves_every_call_and_converges():
    """Online mode: every call returns the exact product while the lite space
    is measured one candidate per call; once all are measured the shape is
    cached, and turning the mode off leaves the cache in place."""
    import torch
    M, N, K = 96, 256, 384
    A, B = workloads.small_int_operands(4242, 1, M, K, N, "f32")
    R = oracle.matmul(A, B)
    dA, dB = dev(A), dev(B)
    nj.nnjit_cache_clear()
    prev = nj.nnjit_set_online(True)
    try:
        calls, states = 0, []
        for calls in range(1, 400):
            C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda:0")
            nj.matmul(dA, dB, C)
            assert np.array_equal(host(C), R), f"call {calls}"      # host() synchronises
            st = nj.nnjit_online_status(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)
            states.append(st)
            if st["state"] == "tuned":
                break
        assert states[-1]["state"] == "tuned", states[-1]
        first = states[0]
        assert first["state"] == "online" and first["total"] >= 8
        assert calls >= first["total"]                 # one candidate per call at most
        measured = [s["measured"] for s in states if s["state"] == "online"]
        assert measured == sorted(measured)           # progress is monotone
        cfg = nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)
        lite, _, _, _ = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)
        assert cfg in lite and cfg == states[-1]["registered"]
        ranked = nj.nnjit_cached_ranked(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)
        assert ranked[0][0] == cfg
    finally:
        nj.nnjit_set_online(prev)
    # later calls use the cached configuration
    C = torch.empty((M, N), dtype=torch.float32, device="cuda:0")
    nj.matmul(dA, dB, C)
    assert np.array_equal(host(C), R)
    nj.nnjit_cache_clear()


def test_concurrent_host_threads_on_own_streams():
    """Four host threads, each on its own stream, alternate default-config
    calls and a forced split-K configuration (each stream's own scratch in use
    at once) while a fifth thread tunes another shape: every result is the
    oracle's exact sum (small integers)."""
    import threading
    import torch
    cfg = next(c for c in nj.configs()
               if c["family"] == "gemm_f32" and c["vec"] == 16 and c["split"] == 4 and c["Mt"] <= 64)
    shapes = [(96, 136, 264), (64, 200, 512), (130, 72, 320), (48, 256, 400)]
    results, errors = {}, []

    def worker(t):
        try:
            M, N, K = shapes[t]
            A, B = workloads.small_int_operands(9100 + t, 1, M, K, N, "f32")
            R = oracle.matmul(A, B)
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                dA = torch.from_numpy(A).to("cuda:0")
                dB = torch.from_numpy(B).to("cuda:0")
                ok = True
                for it in range(16):
                    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda:0")
                    nj.matmul(dA, dB, C, stream=s, cfg=cfg["id"] if it % 2 else None)
                    s.synchronize()
                    ok = ok and np.array_equal(C.cpu().numpy().astype(np.float64), R)
            results[t] = ok
        except Exception as e:   # reported below
            errors.append(repr(e))

    def tuner():
        try:
            nj.check(nj.nnjit_tune(256, 512, 1024, nj.NNJIT_F32))
        except Exception as e:
            errors.append(repr(e))

    nj.matmul(dev(np.ones((4, 8), np.float32)), dev(np.ones((8, 8), np.float32)))   # device state initialised
    torch.cuda.synchronize()
    threads = [threading.Thread(target=worker, args=(t,)) for t in range(4)] + [threading.Thread(target=tuner)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not errors, errors
    assert results == {0: True, 1: True, 2: True, 3: True}


def test_graph_replay_after_scratch_growth():
    """A graph captured on a stream keeps the split-K scratch it was captured
    with: a larger split-K call on the same stream afterwards grows the
    scratch (the old buffer is retired, not freed), and every replay of the
    earlier graph, interleaved with further large calls, still gives the
    oracle's exact sums."""
    import torch
    cfg = next(c for c in nj.configs()
               if c["family"] == "gemm_f32" and c["vec"] == 16 and c["split"] == 4 and not c.get("direct"))
    small = (64, 192, 512)
    large = (256, 1024, 1024)
    cases = {}
    for tag, (M, N, K) in (("small", small), ("large", large)):
        A, B = workloads.small_int_operands(5150 + M, 1, M, K, N, "f32")
        cases[tag] = (M, N, K, dev(A), dev(B), oracle.matmul(A, B))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        outs = {t: torch.full((v[0], v[1]), float("nan"), dtype=torch.float32, device="cuda:0")
                for t, v in cases.items()}

    def call(tag):
        M, N, K, dA, dB, _ = cases[tag]
        return nj.nnjit_matmul_config(cfg["id"], 1, M, N, K, dA, K, 0, dB, N, 0, outs[tag], N, 0, nj.NNJIT_F32,
                                      side)

    with torch.cuda.stream(side):
        assert call("small") == nj.NNJIT_OK   # the stream's scratch sized for the small product
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        assert call("small") == nj.NNJIT_OK
    with torch.cuda.stream(side):
        assert call("large") == nj.NNJIT_OK   # grows the scratch past the captured buffer
    torch.cuda.synchronize()
    assert np.array_equal(host(outs["large"]), cases["large"][5])
    for rep in range(4):
        outs["small"].fill_(float("nan"))
        outs["large"].fill_(float("nan"))
        torch.cuda.synchronize()
        with torch.cuda.stream(side):
            g.replay()
            assert call("large") == nj.NNJIT_OK
        torch.cuda.synchronize()
        assert np.array_equal(host(outs["small"]), cases["small"][5]), f"replay {rep}"
        assert np.array_equal(host(outs["large"]), cases["large"][5]), f"large call {rep}"


def test_product_served_from_loaded_database(tmp_path):
    """A shape tuned in one session, saved to the kernel database, is served
    after a cache clear and a load from that file: the dispatch runs the
    stored configuration and its result meets the acceptance bar against
    the oracle (workload values, every element)."""
    name, index = "t5_large_layer_b4s256_f32", 5
    op = workloads.workload(name)[index]
    nj.nnjit_cache_clear()
    cfg = nj.check(nj.nnjit_tune(op.M, op.N, op.K, nj.NNJIT_F32))
    path = tmp_path / "db.txt"
    assert nj.check(nj.nnjit_cache_save(str(path))) == 1
    nj.nnjit_cache_clear()
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K) == nj.NNJIT_ENOCFG
    assert nj.check(nj.nnjit_cache_load(str(path))) == 1
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, op.M, op.N, op.K) == cfg
    A, B = workloads.op_inputs(name, index)
    dA, dB = dev(A), dev(B)
    C = host(nj.matmul(dA, dB))
    assert np.array_equal(C, host(nj.matmul(dA, dB, cfg=cfg)))     # the stored configuration ran
    res = accept.check(C, oracle.matmul(A, B), A, B, "f32")
    assert res["ok"], res
    nj.nnjit_cache_clear()


def test_online_failing_candidate_falls_back(monkeypatch):
    """Online mode with a candidate that cannot launch: that call's product is
    computed by the registered configuration (exact sums), the candidate is
    never registered, and the shape still ends tuned."""
    import torch
    M, N, K = 96, 256, 384
    lite, _, _, _ = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)
    bad = lite[1]
    A, B = workloads.small_int_operands(4343, 1, M, K, N, "f32")
    R = oracle.matmul(A, B)
    dA, dB = dev(A), dev(B)
    monkeypatch.setenv("NNJIT_FAULT_CONFIG", str(bad))
    nj.nnjit_cache_clear()   # the library reads its environment here
    prev = nj.nnjit_set_online(True)
    try:
        for calls in range(1, 400):
            C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda:0")
            nj.matmul(dA, dB, C)
            assert np.array_equal(host(C), R), f"call {calls}"
            st = nj.nnjit_online_status(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)
            if st["state"] == "tuned":
                break
        assert st["state"] == "tuned"
        cfg = nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)
        assert cfg != bad
        assert bad not in [c for c, _ in nj.nnjit_cached_ranked(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)]
    finally:
        nj.nnjit_set_online(prev)
        monkeypatch.delenv("NNJIT_FAULT_CONFIG")
        nj.nnjit_cache_clear()


def test_tune_does_not_block_dispatch_on_other_threads():
    """While one thread tunes a large shape (hundreds of milliseconds),
    another thread's calls return without waiting for it; their results are
    exact."""
    import threading
    import torch
    nj.nnjit_cache_clear()
    M, N, K = 64, 128, 256
    A, B = workloads.small_int_operands(4444, 1, M, K, N, "f32")
    R = oracle.matmul(A, B)
    dA, dB = dev(A), dev(B)
    C = nj.matmul(dA, dB)                  # device state and this shape's default set up
    torch.cuda.synchronize()
    started, errors = threading.Event(), []

    def tuner():
        started.set()
        try:
            nj.check(nj.nnjit_tune(512, 32000, 4096, nj.NNJIT_F32))
        except Exception as e:   # reported below
            errors.append(repr(e))

    th = threading.Thread(target=tuner)
    th.start()
    started.wait()
    import time
    time.sleep(0.05)                       # the tune is under way (scratch set-up, candidates)
    alive_before = th.is_alive()
    for _ in range(20):
        nj.matmul(dA, dB, C)
    alive_after = th.is_alive()
    th.join(timeout=120)
    assert not errors, errors
    assert np.array_equal(host(C), R)
    st_tuned = nj.nnjit_cached_config(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, 512, 32000, 4096)
    assert st_tuned >= 0
    if alive_before:
        assert alive_after, "the calls waited for the tune to finish"
    nj.nnjit_cache_clear()


def test_tune_trace_agrees_with_stats_and_lite_space():
    """The evaluation trace of a tune -- one entry per first-pass candidate,
    in the lite space's order: its id, its per-launch time (-1 when aborted
    or failed) and the milliseconds since the call began -- agrees with the
    call's statistics; the returned count is the full length whatever the
    cap; a cache hit evaluates nothing."""
    import ctypes
    nj.nnjit_cache_clear()
    M, N, K = 256, 1024, 512
    cfg = nj.nnjit_tune(M, N, K, nj.NNJIT_F32)
    assert cfg >= 0, nj.nnjit_last_error()
    st = nj.nnjit_last_tune_stats_ex()
    tr = nj.nnjit_last_tune_trace(4096)
    assert len(tr) >= 2
    assert len(tr) == st["n_timed"] + st["n_aborted"] + st["n_failed"]
    ids = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, M, N, K)[0]
    assert [t[0] for t in tr] == ids[:len(tr)]
    timed = [t for t in tr if t[1] >= 0]
    assert len(timed) == st["n_timed"] and all(t[1] > 0 for t in timed)
    at = [t[2] for t in tr]
    assert at == sorted(at) and 0 <= at[0] and at[-1] <= st["wall_ms"]
    assert st["chosen"] == cfg and cfg in {t[0] for t in timed}
    a, u, m = (ctypes.c_int * 2)(), (ctypes.c_double * 2)(), (ctypes.c_double * 2)()
    assert nj.load().nnjit_last_tune_trace(a, u, m, 2) == len(tr)
    assert [(a[i], u[i], m[i]) for i in range(2)] == tr[:2]
    assert nj.nnjit_tune(M, N, K, nj.NNJIT_F32) == cfg
    assert nj.nnjit_last_tune_trace() == []
    assert nj.nnjit_last_tune_stats_ex()["cache_hit"] == 1
