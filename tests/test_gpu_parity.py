"""GPU parity of the HIP path against the CPU oracle, through the C-ABI.

* every configuration id, forced, on small-integer operands at ragged shapes
  spanning several tiles: bit-exact (all partial sums are exact in fp32, so
  any summation order gives the oracle's value), and run twice: identical;
* every workload shape at full size, tuned, on the workload's own value
  distributions: fp32 within rel-Frobenius 1e-5 and |err| <= 2e-6 K max|A|
  max|B| per element; fp16 inputs within rel-Frobenius 2e-3 -- over every
  element of the output; and the same shape through the same tuned
  configuration on small-integer operands: bit-exact over every element;
* edge cases: K = 0, empty operands, padded leading dimensions, batch strides
  with gaps, misaligned operands (element-load fallback), M = 1 batches;
* metamorphic relations: power-of-two scaling and batch slices are
  bit-exact, (B^T A^T)^T matches within tolerance.
"""
import numpy as np
import pytest

import oracle
from oracle import accept
import paper_2309_08978_amd as nj
import workloads
from tests.gpu_util import dev, host, gpu_matmul, kind_of, dtype_code

pytestmark = pytest.mark.gpu

FAMILY_DTYPE = {"gemm_f32": "f32", "gemm_f16": "f16", "gemv_f32": "f32", "gemv_f16": "f16"}


def _family_shapes(family: str, vec: bool):
    """(batch, M, N, K) used to pin every configuration of a family.  Vector
    (16-byte) configurations need N and K multiples of 8 elements; the
    element-load ones get fully ragged shapes."""
    gemv = family.startswith("gemv")
    if gemv:
        return (1, 1, 1032, 997) if vec else (1, 1, 1027, 997)
    return (2, 291, 264, 200) if vec else (2, 291, 259, 197)


@pytest.fixture(scope="module")
def all_configs():
    nj.load()
    return nj.configs()


def _int_case(family, vec, seed):
    batch, M, N, K = _family_shapes(family, vec)
    dt = FAMILY_DTYPE[family]
    A, B = workloads.small_int_operands(seed, batch, M, K, N, dt)
    R = oracle.matmul(A, B)
    return A, B, R


@pytest.mark.parametrize("family", ["gemm_f32", "gemm_f16", "gemv_f32", "gemv_f16"])
def test_every_config_bit_exact_small_integers(all_configs, family):
    import torch
    cases = {}
    n = 0
    for c in all_configs:
        if c["family"] != family:
            continue
        vec = c["vec"] == 16
        if vec not in cases:
            cases[vec] = _int_case(family, vec, 1000 + int(vec))
        A, B, R = cases[vec]
        dA, dB = dev(A), dev(B)
        shape = R.shape
        outs = []
        for rep in range(2):
            C = torch.full(shape, float("nan"), dtype=torch.float32, device="cuda:0")
            if A.ndim == 2:
                nj.matmul(dA, dB, C, cfg=c["id"])
            else:
                nj.batched_matmul(dA, dB, C, cfg=c["id"])
            outs.append(host(C))
        assert np.array_equal(outs[0], R), f"config {c['id']} {c['name']} split={c['split']} differs from the oracle"
        assert np.array_equal(outs[0], outs[1]), f"config {c['id']} not deterministic"
        n += 1
    assert n > 0
    print(f"{family}: {n} configurations bit-exact", flush=True)


@pytest.mark.parametrize("K", [8, 16, 40])
def test_direct_copy_configs_short_k(all_configs, K):
    """Direct-copy configurations (per-wave K slices, LDS stages) when K is
    shorter than one slab per wave or stage: idle waves, partly empty
    pipelines and a ragged last slab still give the oracle's exact sums."""
    import torch
    n = 0
    for family in ("gemm_f32", "gemm_f16"):
        A, B = workloads.small_int_operands(77 + K, 1, 70, K, 136, FAMILY_DTYPE[family])
        R = oracle.matmul(A, B)
        dA, dB = dev(A), dev(B)
        for c in all_configs:
            if c["family"] != family or not c.get("direct"):
                continue
            C = torch.full(R.shape, float("nan"), dtype=torch.float32, device="cuda:0")
            nj.matmul(dA, dB, C, cfg=c["id"])
            assert np.array_equal(host(C), R), f"config {c['id']} {c['name']} split={c['split']} K={K}"
            n += 1
    assert n > 0



@pytest.mark.parametrize("K", [1024, 1064])
def test_direct_copy_configs_long_k(all_configs, K):
    """Direct-copy configurations, every split, with K long enough that each
    wave (or workgroup) runs the branch-free main loop over whole K slabs
    with unchecked copies before the checked loop takes the rest: whole slabs
    only (K = 1024) and a ragged last slab (K = 1064), with M and N ragged
    against every tile (rows and columns past the edge are read from row /
    column 0 in the main loop and never stored).  Small integers: the
    oracle's exact sums."""
    import torch
    n = 0
    for family in ("gemm_f32", "gemm_f16"):
        A, B = workloads.small_int_operands(5150 + K, 1, 70, K, 136, FAMILY_DTYPE[family])
        R = oracle.matmul(A, B)
        dA, dB = dev(A), dev(B)
        for c in all_configs:
            if c["family"] != family or not c.get("direct"):
                continue
            C = torch.full(R.shape, float("nan"), dtype=torch.float32, device="cuda:0")
            nj.matmul(dA, dB, C, cfg=c["id"])
            assert np.array_equal(host(C), R), f"config {c['id']} {c['name']} split={c['split']} K={K}"
            n += 1
    assert n > 0
    print(f"K={K}: {n} direct-copy configurations bit-exact", flush=True)

WL_OPS = [(name, i) for name in workloads.WORKLOADS for i in range(len(workloads.workload(name)))
          if workloads.workload(name)[i].dtype != workloads.Q4]   # 4-bit GEMV: tests/test_gpu_q4.py


def _tune_op(op) -> int:
    dt = dtype_code(op.dtype)
    if op.batch == 1:
        cfg = nj.check(nj.nnjit_tune(op.M, op.N, op.K, dt))
    else:
        cfg = nj.check(nj.nnjit_tune_batched(op.batch, op.M, op.N, op.K, dt))
    lite, _, _, _ = nj.nnjit_lite_space(kind_of(op.batch, op.M), dt, op.batch, op.M, op.N, op.K)
    assert cfg in lite
    return cfg


@pytest.mark.parametrize("name,index", WL_OPS, ids=[f"{n}-{workloads.workload(n)[i].name}" for n, i in WL_OPS])
def test_workload_shape_parity(name, index):
    """The tuned configuration of a workload product, on the workload's own
    values at full size, against the oracle over every output element."""
    import torch
    op = workloads.workload(name)[index]
    A, B = workloads.op_inputs(name, index)
    dt = dtype_code(op.dtype)
    cfg = _tune_op(op)
    st = nj.nnjit_last_tune_stats_ex()
    print(f"{name}/{op.name}: tuned -> {nj.nnjit_config_info(cfg)} | {st['best_us']:.2f} us, "
          f"lite {st['n_lite']}, timed {st['n_timed']}, tune {st['wall_ms']:.0f} ms", flush=True)
    C = gpu_matmul(A, B)  # dispatch through the tuned cache
    assert nj.nnjit_cached_config(kind_of(op.batch, op.M), dt, op.batch, op.M, op.N, op.K) == cfg
    R = oracle.matmul(A, B)
    res = accept.check(C, R, A, B, op.dtype)
    print(f"   all {C.size} elements: rel_fro={res['rel_fro']:.3e} max_err={res['max_err']:.3e} "
          f"bound={res['elt_bound']:.3e}", flush=True)
    assert res["ok"], res
    if op.dtype == "f16":
        # informational: fp16 x fp16 products are exact in fp32, so the fp32 bar usually holds too
        print(f"   (fp32 bar on fp16 inputs: {accept.check(C, R, A, B, 'f32')['ok']})", flush=True)
    del C
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,index", WL_OPS, ids=[f"{n}-{workloads.workload(n)[i].name}" for n, i in WL_OPS])
def test_workload_shape_small_int_bit_exact(name, index):
    """The same full-size shape through the same tuned configuration (with
    its split factor and tile grid) on operands in {-8..8}: every partial
    sum is an integer below 2^24 (K <= 11 008), so the result is exact in
    fp32 whatever the summation order and must equal the oracle's over every
    element."""
    import torch
    op = workloads.workload(name)[index]
    cfg = _tune_op(op)
    A, B = workloads.small_int_operands(90000 + 97 * index + len(name), op.batch, op.M, op.K, op.N, op.dtype)
    C = gpu_matmul(A, B)
    assert nj.nnjit_cached_config(kind_of(op.batch, op.M), dtype_code(op.dtype), op.batch, op.M, op.N, op.K) == cfg
    R = oracle.matmul(A, B)
    bad = np.argwhere(C != R)
    assert bad.size == 0, (f"{name}/{op.name} config {nj.nnjit_config_info(cfg)}: {len(bad)} of {C.size} "
                           f"elements differ, first at {tuple(bad[0])}")
    print(f"{name}/{op.name}: {C.size} elements bit-exact on {nj.nnjit_config_info(cfg).split()[2]}", flush=True)
    del C
    torch.cuda.empty_cache()


# ------------------------------------------------------------------ edge cases

@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_k_zero_writes_zeros(dt):
    import torch
    tdt = torch.float16 if dt == "f16" else torch.float32
    for (b, M, N) in [(1, 37, 45), (1, 1, 64), (3, 17, 9)]:
        A = torch.empty((b, M, 0), dtype=tdt, device="cuda:0")
        B = torch.empty((b, 0, N), dtype=tdt, device="cuda:0")
        C = torch.full((b, M, N), float("nan"), device="cuda:0")
        if b == 1:
            nj.matmul(A[0], B[0], C[0])
        else:
            nj.batched_matmul(A, B, C)
        assert np.array_equal(host(C), np.zeros((b, M, N)))


def test_empty_shapes_are_noops():
    import torch
    C = torch.full((4, 5), 7.0, device="cuda:0")
    A = torch.ones((4, 3), device="cuda:0")
    B = torch.ones((3, 5), device="cuda:0")
    assert nj.nnjit_matmul(0, 5, 3, A, 3, B, 5, C, 5, 0, None) == 0
    assert nj.nnjit_matmul(4, 0, 3, A, 3, B, 5, C, 5, 0, None) == 0
    assert nj.nnjit_batched_matmul(0, 4, 5, 3, A, 3, 12, B, 5, 15, C, 5, 20, 0, None) == 0
    assert np.all(host(C) == 7.0)


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_padded_leading_dims_and_batch_gaps(dt):
    import torch
    b, M, N, K = 3, 70, 136, 96
    A, B = workloads.small_int_operands(77, b, M, K, N, dt)
    R = oracle.matmul(A, B)
    tdt = torch.float16 if dt == "f16" else torch.float32
    lda, ldb, ldc = K + 8, N + 16, N + 5
    sA, sB, sC = M * lda + 64, K * ldb + 40, M * ldc + 11
    bufA = torch.zeros(b * sA, dtype=tdt, device="cuda:0")
    bufB = torch.zeros(b * sB, dtype=tdt, device="cuda:0")
    bufC = torch.full((b * sC,), -3.0, device="cuda:0")
    for i in range(b):
        bufA[i * sA:i * sA + M * lda].view(M, lda)[:, :K] = dev(A[i])
        bufB[i * sB:i * sB + K * ldb].view(K, ldb)[:, :N] = dev(B[i])
    rc = nj.nnjit_batched_matmul(b, M, N, K, bufA, lda, sA, bufB, ldb, sB, bufC, ldc, sC, dtype_code(dt), None)
    assert rc == 0, nj.nnjit_last_error()
    hc = host(bufC)
    for i in range(b):
        Ci = hc[i * sC:i * sC + M * ldc].reshape(M, ldc)
        assert np.array_equal(Ci[:, :N], R[i])
        assert np.all(Ci[:, N:] == -3.0)  # padding untouched
        if i + 1 < b:
            assert np.all(hc[i * sC + M * ldc:(i + 1) * sC] == -3.0)


@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("M", [1, 45])
def test_misaligned_operands_use_fallback(dt, M):
    import torch
    N, K = 200, 96
    A, B = workloads.small_int_operands(78, 1, M, K, N, dt)
    R = oracle.matmul(A, B)
    tdt = torch.float16 if dt == "f16" else torch.float32
    bA = torch.zeros(M * K + 1, dtype=tdt, device="cuda:0")
    bB = torch.zeros(K * N + 1, dtype=tdt, device="cuda:0")
    bA[1:] = dev(A).reshape(-1)
    bB[1:] = dev(B).reshape(-1)
    C = torch.full((M, N), float("nan"), device="cuda:0")
    rc = nj.nnjit_matmul(M, N, K, bA.data_ptr() + bA.element_size(), K, bB.data_ptr() + bB.element_size(), N,
                         C, N, dtype_code(dt), None)
    assert rc == 0, nj.nnjit_last_error()
    assert np.array_equal(host(C), R)


def test_batch_of_row_vectors():
    A, B = workloads.small_int_operands(79, 5, 1, 300, 260, "f32")
    assert np.array_equal(gpu_matmul(A, B), oracle.matmul(A, B))


def test_forced_config_mismatch_is_einval(all_configs):
    import torch
    A = torch.ones((4, 8), device="cuda:0")
    B = torch.ones((8, 8), device="cuda:0")
    C = torch.empty((4, 8), device="cuda:0")
    gemv = next(c["id"] for c in all_configs if c["family"] == "gemv_f32")
    f16 = next(c["id"] for c in all_configs if c["family"] == "gemm_f16")
    assert nj.nnjit_matmul_config(gemv, 1, 4, 8, 8, A, 8, 0, B, 8, 0, C, 8, 0, 0, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_matmul_config(f16, 1, 4, 8, 8, A, 8, 0, B, 8, 0, C, 8, 0, 0, None) == nj.NNJIT_EINVAL
    vec = next(c["id"] for c in all_configs if c["family"] == "gemm_f32" and c["vec"] == 16)
    rc = nj.nnjit_matmul_config(vec, 1, 4, 8, 8, A.data_ptr() + 4, 8, 0, B, 8, 0, C, 8, 0, 0, None)
    assert rc == nj.NNJIT_EINVAL


# --------------------------------------------------------------- metamorphic

def test_power_of_two_scaling_bit_exact():
    op = workloads.workload("bart_base_layer_seq128_f32")[2]
    A, B = workloads.op_inputs("bart_base_layer_seq128_f32", 2)
    C1 = gpu_matmul(A, B)
    C2 = gpu_matmul((A * np.float32(8)).astype(np.float32), B)
    assert np.array_equal(C2, 8 * C1), op.name


def test_batch_slices_match_single_products(all_configs):
    A, B = workloads.random_operands(80, 4, 96, 136, 72, "f32")
    for c in all_configs:
        if c["family"] != "gemm_f32" or c["vec"] != 16 or c["split"] not in (1, 4):
            continue
        Cb = gpu_matmul(A, B, cfg=c["id"])
        for i in range(4):
            assert np.array_equal(Cb[i], gpu_matmul(A[i], B[i], cfg=c["id"])), c["name"]


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_transpose_identity(dt):
    A, B = workloads.random_operands(81, 1, 160, 256, 200, dt)
    C = gpu_matmul(A, B)
    Ct = gpu_matmul(np.ascontiguousarray(B.T), np.ascontiguousarray(A.T)).T
    R = oracle.matmul(A, B)
    assert accept.check(C, R, A, B, dt)["ok"]
    assert accept.check(Ct, R, A, B, dt)["ok"]


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_batch_beyond_one_launch(all_configs, dt):
    """70 001 batch slices: more than the 65 535 a launch's grid.z holds, so
    the batch is cut into several launches (and, with split-K, several
    reductions over the matching slices of the scratch).  Small integers:
    bit-exact against the oracle, on the default configuration and on a
    forced split-K configuration."""
    import torch
    batch, M, N, K = 70001, 3, 8, 40
    A, B = workloads.small_int_operands(31337, batch, M, K, N, dt)
    R = oracle.matmul(A, B)
    dA, dB = dev(A), dev(B)
    C = nj.batched_matmul(dA, dB)
    assert np.array_equal(host(C), R)
    fam = "gemm_f16" if dt == "f16" else "gemm_f32"
    cfg = next(c for c in all_configs if c["family"] == fam and c["vec"] == 16 and c["split"] == 4 and c["Mt"] <= 64)
    C2 = torch.full(R.shape, float("nan"), dtype=torch.float32, device="cuda:0")
    nj.batched_matmul(dA, dB, C2, cfg=cfg["id"])
    assert np.array_equal(host(C2), R), f"config {cfg['name']} split={cfg['split']}"


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_gemv_split_k_back_to_back_and_replayed(all_configs, dt):
    """Split-K GEMV: launches of different configurations, splits and column
    segment counts back to back on one stream (no host synchronisation
    between them, each reduction reading the scratch its own GEMV just
    wrote), then a graph of three of them replayed four times: every result
    is the oracle's exact sum (small integers)."""
    import torch
    fam = "gemv_" + dt
    split = [c for c in all_configs if c["family"] == fam and c["vec"] == 16 and c["split"] > 1]
    assert split
    picks = split[:: max(1, len(split) // 8)][:8]
    shapes = [(1, 2056, 4096), (1, 1032, 997), (1, 8192, 3000), (1, 264, 5000)]   # (M, N, K)
    cases = []
    for i, c in enumerate(picks):
        M, N, K = shapes[i % len(shapes)]
        A, B = workloads.small_int_operands(7300 + i, 1, M, K, N, dt)
        cases.append((c, dev(A), dev(B), oracle.matmul(A, B)))
    outs = [torch.full(R.shape, float("nan"), dtype=torch.float32, device="cuda:0") for _, _, _, R in cases]
    for (c, dA, dB, _), C in zip(cases, outs):
        nj.matmul(dA, dB, C, cfg=c["id"])
    torch.cuda.synchronize()
    for (c, _, _, R), C in zip(cases, outs):
        assert np.array_equal(host(C), R), f"config {c['name']} split={c['split']}"

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    trio = cases[:3]

    def step():
        for (c, dA, dB, _), C in zip(trio, outs):
            nj.matmul(dA, dB, C, stream=side, cfg=c["id"])
    with torch.cuda.stream(side):
        step()   # scratch and counters of the side stream allocated outside capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        step()
    for rep in range(4):
        for C in outs:
            C.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for (c, _, _, R), C in zip(trio, outs):
            assert np.array_equal(host(C), R), f"replay {rep}: config {c['name']} split={c['split']}"


@pytest.mark.parametrize("family", ["gemm_f32", "gemm_f16"])
def test_tile_order_groups_cover_every_tile(all_configs, family, monkeypatch):
    """The tile order runs in groups of G tile rows (NNJIT_GROUP_M forces G):
    for every G, including ones that do not divide the tile rows and the
    plain column order, each tile is computed exactly once -- the output
    (NaN-filled first) is the oracle's exact sum, with split-K and batch."""
    import torch
    batch, M, N, K = 2, 1000, 520, 96
    A, B = workloads.small_int_operands(6061, batch, M, K, N, FAMILY_DTYPE[family])
    R = oracle.matmul(A, B)
    dA, dB = dev(A), dev(B)
    # one 64-row configuration of each kernel of the family, unsplit and split 2
    prefixes = (("gemm_f32_", "gemm_f32w_", "gemm_f32t_") if family == "gemm_f32" else ("gemm_f16_", "gemm_f16t_"))
    picks = []
    for pre in prefixes:
        for split in (1, 2):
            picks += [c for c in all_configs if c["family"] == family and c["vec"] == 16 and c["Mt"] == 64
                      and c["name"].startswith(pre) and c["split"] == split][:1]
    assert len(picks) == 2 * len(prefixes), [c["name"] for c in picks]
    try:
        for G in ("1", "3", "4", "5", "16", "64"):
            monkeypatch.setenv("NNJIT_GROUP_M", G)
            nj.nnjit_cache_clear()   # the library reads its environment here
            for c in picks:
                C = torch.full(R.shape, float("nan"), dtype=torch.float32, device="cuda:0")
                nj.batched_matmul(dA, dB, C, cfg=c["id"])
                assert np.array_equal(host(C), R), f"G={G} config {c['name']} split={c['split']}"
    finally:
        monkeypatch.delenv("NNJIT_GROUP_M")
        nj.nnjit_cache_clear()


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_random_shapes_bit_exact(all_configs, dt):
    """Seeded random shapes (batch 1-3, M 1-300, N 8-520 in steps of 8 or any,
    K 1-1500): the default configuration and two random configurations of the
    family that accept the operands all give the oracle's exact sums (small
    integers), covering slab, split and tile boundaries no fixed case hits."""
    import torch
    rng = np.random.default_rng(20240 + (dt == "f16"))
    fam = "gemm_" + dt
    n = 0
    for t in range(24):
        batch = int(rng.integers(1, 4))
        M = int(rng.integers(1, 301))
        vec = bool(rng.integers(0, 2))
        N = int(rng.integers(1, 66)) * 8 if vec else int(rng.integers(1, 521))
        K = int(rng.integers(1, 188)) * 8 if vec else int(rng.integers(1, 1501))
        if M == 1:
            M = 2   # M = 1 is the GEMV kind, covered elsewhere
        A, B = workloads.small_int_operands(30000 + t, batch, M, K, N, dt)
        R = oracle.matmul(A, B)
        dA, dB = dev(A), dev(B)
        mm = nj.matmul if A.ndim == 2 else nj.batched_matmul
        C = mm(dA, dB)
        assert np.array_equal(host(C), R), f"default: batch={batch} M={M} N={N} K={K}"
        want16 = vec and (K * (2 if dt == "f16" else 4)) % 16 == 0 and (N * (2 if dt == "f16" else 4)) % 16 == 0
        pool = [c for c in all_configs if c["family"] == fam and (c["vec"] == 16) == want16]
        for c in rng.choice(pool, size=2, replace=False):
            C = torch.full(R.shape, float("nan"), dtype=torch.float32, device="cuda:0")
            mm(dA, dB, C, cfg=int(c["id"]))
            assert np.array_equal(host(C), R), f"{c['name']} split={c['split']}: batch={batch} M={M} N={N} K={K}"
            n += 1
    print(f"{dt}: {n} forced random-shape runs bit-exact", flush=True)


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_random_gemv_shapes_bit_exact(all_configs, dt):
    """Seeded random M = 1 shapes (N 1-9000, K 1-6000, aligned or not): the
    default configuration and three random GEMV configurations that accept
    the operands (any split) give the oracle's exact sums (small integers)."""
    import torch
    rng = np.random.default_rng(40960 + (dt == "f16"))
    fam = "gemv_" + dt
    n = 0
    for t in range(20):
        vec = bool(rng.integers(0, 2))
        N = int(rng.integers(1, 1126)) * 8 if vec else int(rng.integers(1, 9001))
        K = int(rng.integers(1, 6001))
        A, B = workloads.small_int_operands(50000 + t, 1, 1, K, N, dt)
        R = oracle.matmul(A, B)
        dA, dB = dev(A), dev(B)
        C = nj.matmul(dA, dB)
        assert np.array_equal(host(C), R), f"default: N={N} K={K}"
        pool = [c for c in all_configs if c["family"] == fam and (c["vec"] == 16) == vec]
        for c in rng.choice(pool, size=3, replace=False):
            C = torch.full(R.shape, float("nan"), dtype=torch.float32, device="cuda:0")
            nj.matmul(dA, dB, C, cfg=int(c["id"]))
            assert np.array_equal(host(C), R), f"{c['name']} split={c['split']}: N={N} K={K}"
            n += 1
    print(f"{dt}: {n} forced random GEMV runs bit-exact", flush=True)


@pytest.mark.parametrize("shape", [(300, 520, 1000), (512, 1024, 2048), (64, 128, 4100), (1000, 264, 72),
                                   (130, 64, 16), (257, 1032, 520)])
def test_stream_k_configs_bit_exact(all_configs, shape):
    """Every stream-K configuration (the tiles' K slabs cut evenly over one
    workgroup per resident slot; shared tiles summed by the fix-up kernel)
    on ragged shapes -- tiles shared by two or more workgroups, workgroups
    spanning several tiles, K not a multiple of the slab -- gives the
    oracle's exact sums (small integers), twice in a row; a batched call
    forced onto it runs tiled."""
    import torch
    M, N, K = shape
    A, B = workloads.small_int_operands(7700 + M + K, 1, M, K, N, "f32")
    R = oracle.matmul(A, B)
    dA, dB = dev(A), dev(B)
    sk = [c for c in all_configs if c["family"] == "gemm_f32" and c["split"] == 0]
    assert sk
    for c in sk:
        for rep in range(2):
            C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda:0")
            nj.matmul(dA, dB, C, cfg=c["id"])
            assert np.array_equal(host(C), R), f"{c['name']} stream-K {shape} rep {rep}"
    c = sk[0]
    A3, B3 = workloads.small_int_operands(7800, 3, 40, 96, 136, "f32")
    C3 = torch.full((3, 40, 136), float("nan"), dtype=torch.float32, device="cuda:0")
    nj.batched_matmul(dev(A3), dev(B3), C3, cfg=c["id"])
    assert np.array_equal(host(C3), oracle.matmul(A3, B3))
