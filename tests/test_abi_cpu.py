"""Host-side tests of the C-ABI library (no GPU): it loads, exports every
entry point include/nnjit.h declares, validates arguments before touching
HIP, and its lite-space builder follows the Table 1 resource model and
heuristics of the paper (Sec. 5.2)."""
import json
import os
import re

import pytest

import paper_2309_08978_amd as nj
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "nnjit.h")


@pytest.fixture(scope="module")
def lib():
    return nj.load(build_if_missing=True)


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char \*)\s*(nnjit_\w+)\s*\(", src, re.M)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(nj.EXPORTED)


def test_validation_without_gpu(lib):
    # bad arguments are reported before any HIP call
    assert nj.nnjit_matmul(4, 4, 4, 1, 4, 2, 4, 3, 4, 9, None) == nj.NNJIT_EDTYPE
    assert nj.nnjit_matmul(-1, 4, 4, 1, 4, 2, 4, 3, 4, 0, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_matmul(4, 4, 4, 1, 3, 2, 4, 3, 4, 0, None) == nj.NNJIT_EINVAL  # lda < K
    assert nj.nnjit_matmul(4, 4, 4, 1, 4, 2, 3, 3, 4, 0, None) == nj.NNJIT_EINVAL  # ldb < N
    assert nj.nnjit_matmul(4, 4, 4, 1, 4, 2, 4, 3, 3, 0, None) == nj.NNJIT_EINVAL  # ldc < N
    assert nj.nnjit_matmul(4, 4, 4, None, 4, 2, 4, 3, 4, 0, None) == nj.NNJIT_EINVAL
    assert "A is NULL" in nj.nnjit_last_error()
    assert nj.nnjit_batched_matmul(2, 4, 4, 4, 1, 4, -1, 2, 4, 16, 3, 4, 16, 0, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_matmul(1 << 31, 4, 4, 1, 4, 2, 4, 3, 4, 0, None) == nj.NNJIT_EINVAL
    # empty products are no-ops that never touch the GPU
    assert nj.nnjit_matmul(0, 4, 4, None, 4, 2, 4, None, 4, 0, None) == nj.NNJIT_OK
    assert nj.nnjit_batched_matmul(0, 4, 4, 4, None, 4, 16, None, 4, 16, None, 4, 16, 0, None) == nj.NNJIT_OK
    assert nj.nnjit_matmul_config(nj.nnjit_num_configs(), 1, 4, 4, 4, 1, 4, 0, 2, 4, 0, 3, 4, 0, 0, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_tune(64, 64, 64, 5) == nj.NNJIT_EDTYPE
    assert nj.nnjit_tune(0, 64, 64, 0) == nj.NNJIT_EINVAL
    # 4-bit GEMV: (N, K, group, x, Wq, ldq, scales, lds, y, stream)
    assert nj.nnjit_gemv_q4(64, 64, 0, 1, 2, 8, 3, 2, 4, None) == nj.NNJIT_EINVAL       # group < 1
    assert nj.nnjit_gemv_q4(64, 64, 32, 1, 2, 7, 3, 2, 4, None) == nj.NNJIT_EINVAL      # ldq < ceil(K/8)
    assert nj.nnjit_gemv_q4(64, 64, 32, 1, 2, 8, 3, 1, 4, None) == nj.NNJIT_EINVAL      # lds < ceil(K/group)
    assert nj.nnjit_gemv_q4(-1, 64, 32, 1, 2, 8, 3, 2, 4, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_gemv_q4(64, 64, 32, 1, None, 8, 3, 2, 4, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_gemv_q4(64, 64, 32, 1, 2, 8, 3, 2, None, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_gemv_q4(0, 64, 32, 1, 2, 8, 3, 2, None, None) == nj.NNJIT_OK       # N == 0: no-op
    assert nj.nnjit_tune_gemv_q4(64, 64, 0) == nj.NNJIT_EINVAL
    cfgs = nj.configs()
    q4 = next(c["id"] for c in cfgs if c["family"] == "gemv_q4")
    f16 = next(c["id"] for c in cfgs if c["family"] == "gemm_f16")
    # a 4-bit configuration is not a MatMul configuration, and the other way round
    assert nj.nnjit_matmul_config(q4, 1, 4, 8, 8, 1, 8, 0, 2, 8, 0, 3, 8, 0, 1, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_gemv_q4_config(f16, 64, 64, 32, 1, 2, 8, 3, 2, 4, None) == nj.NNJIT_EINVAL
    # streaming-read reference: (src, bytes, sink, workgroups, stream)
    assert nj.nnjit_stream_read(16, 24, 32, 8, None) == nj.NNJIT_EINVAL                 # bytes not a multiple of 16
    assert nj.nnjit_stream_read(16, -16, 32, 8, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_stream_read(16, 64, 32, 0, None) == nj.NNJIT_EINVAL                 # no workgroup
    assert nj.nnjit_stream_read(16, 64, 32, (1 << 20) + 1, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_stream_read(8, 64, 32, 8, None) == nj.NNJIT_EINVAL                  # src not 16-byte aligned
    assert nj.nnjit_stream_read(None, 64, 32, 8, None) == nj.NNJIT_EINVAL
    assert nj.nnjit_stream_read(16, 64, None, 8, None) == nj.NNJIT_EINVAL               # no sink
    assert nj.nnjit_stream_read(None, 0, 32, 8, None) == nj.NNJIT_OK                    # nothing to read


def test_tune_stats_forms(lib):
    """The four-pointer statistics call and the full struct agree, and NULL
    outputs are allowed (nothing tuned yet on this thread: zeros)."""
    import ctypes
    assert lib.nnjit_last_tune_stats(None, None, None, None) == nj.NNJIT_OK
    short = nj.nnjit_last_tune_stats()
    full = nj.nnjit_last_tune_stats_ex()
    assert short == {"wall_ms": full["wall_ms"], "n_enum": full["n_enumerated"], "n_pruned": full["n_lite"],
                     "n_timed": full["n_timed"]}
    assert lib.nnjit_last_tune_stats_ex(ctypes.cast(None, ctypes.POINTER(nj.TuneStats))) == nj.NNJIT_EINVAL


def test_binding_rejects_bad_operands(lib):
    """The tensor conveniences refuse, before any library call, operands that
    the entry points would read or write out of bounds."""
    import torch
    f32, f16 = torch.float32, torch.float16
    A = torch.zeros(4, 8)
    B = torch.zeros(8, 6)
    with pytest.raises(TypeError, match="B is"):
        nj.matmul(A, B.to(f16))
    with pytest.raises(TypeError, match="C must be float32"):
        nj.matmul(A, B, torch.zeros(4, 6, dtype=f16))
    with pytest.raises(ValueError, match="C has shape"):
        nj.matmul(A, B, torch.zeros(4, 5))
    with pytest.raises(ValueError, match="inner dimensions"):
        nj.matmul(A, torch.zeros(7, 6))
    with pytest.raises(ValueError, match="rows overlap"):
        nj.matmul(A, torch.zeros(1, 6).expand(8, 6))      # expanded view: row stride 0
    with pytest.raises(ValueError, match="unit stride"):
        nj.matmul(A, torch.zeros(6, 8).t())               # transposed view
    with pytest.raises(ValueError, match="one GPU"):
        nj.matmul(A, B)                                   # host tensors
    Ab, Bb = torch.zeros(3, 4, 8), torch.zeros(3, 8, 6)
    with pytest.raises(ValueError, match="output slices overlap"):
        nj.batched_matmul(Ab, Bb, torch.zeros(4, 6).expand(3, 4, 6))
    with pytest.raises(ValueError, match="batch sizes"):
        nj.batched_matmul(Ab, torch.zeros(2, 8, 6))
    with pytest.raises(ValueError, match="C has shape"):
        nj.batched_matmul(Ab, Bb, torch.zeros(3, 4, 7))
    with pytest.raises(ValueError, match="one GPU"):
        nj.batched_matmul(Ab, Bb)
    # 4-bit GEMV
    x = torch.zeros(64, dtype=f16)
    Wq = torch.zeros(16, 8, dtype=torch.int32)
    S = torch.zeros(16, 2, dtype=f16)
    with pytest.raises(ValueError, match="rows too short"):
        nj.gemv_q4(x, Wq[:, :7], S, 32, 16)
    with pytest.raises(ValueError, match="y must be"):
        nj.gemv_q4(x, Wq, S, 32, 16, y=torch.zeros(15))
    with pytest.raises(ValueError, match="one GPU"):
        nj.gemv_q4(x, Wq, S, 32, 16)


def test_no_gpu_is_ehip_not_abort(lib):
    try:
        import torch
        if torch.cuda.is_available():
            pytest.skip("a GPU is present")
    except ImportError:
        pass
    assert nj.nnjit_matmul(4, 4, 4, 1, 4, 2, 4, 3, 4, 0, None) == nj.NNJIT_EHIP
    assert nj.nnjit_tune(64, 768, 768, 0) == nj.NNJIT_EHIP
    assert nj.nnjit_last_error()


def test_config_table(lib):
    cfgs = nj.configs()
    assert len(cfgs) == nj.nnjit_num_configs() > 100
    assert [c["id"] for c in cfgs] == list(range(len(cfgs)))
    fams = {c["family"] for c in cfgs}
    assert fams == {"gemm_f32", "gemm_f16", "gemv_f32", "gemv_f16", "gemv_q4"}
    p2 = lambda x: x > 0 and (x & (x - 1)) == 0
    for c in cfgs:
        assert c["vec"] <= 16                     # heuristic 1: at most 128-bit accesses
        assert p2(c["split"]) or (c["split"] == 0 and c["family"] == "gemm_f32" and c["direct"] == 1)   # 0: stream-K
        if c["family"].startswith("gemm"):
            for k in ("Mt", "Nt", "Kt"):
                assert p2(c[k]), (c, k)           # heuristic 2: power-of-two tiles
            wm, wn = map(int, c["waves"].split("x"))
            assert c["Mt"] % wm == 0 and c["Nt"] % wn == 0
            assert c["threads"] == 64 * wm * wn * c["kslices"]
        elif c["family"] == "gemv_q4":
            assert p2(c["rows_per_wave"]) and p2(c["kslices"]) and p2(c["threads"]) and c["split"] == 1
            assert c["rows_per_wg"] == c["rows_per_wave"] * (c["threads"] // 64) // c["kslices"]
        else:
            assert p2(c["cols"]) and p2(c["lanes_per_seg"]) and p2(c["threads"])


def test_table1_resources_golden(lib):
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "table1_resources.json")))
    cfg = next(c for c in nj.configs() if c["name"] == g["config_name"] and c["split"] == 1)
    r = nj.nnjit_config_resources(cfg["id"], nj.mi355x_limits())
    assert r == g["expected"]


def test_resource_limits_follow_the_formula(lib):
    d = nj.mi355x_limits()
    for c in nj.configs():
        r = nj.nnjit_config_resources(c["id"], d)
        regs = -(-r["regs_per_lane"] // 8) * 8
        wps = min(8, 512 // regs)
        assert r["waves_per_wg"] == -(-c["threads"] // 64)
        assert r["reg_limit"] == 4 * wps // r["waves_per_wg"]
        # L1Limit: LDS per CU over LDS per workgroup; a workgroup without LDS has no such limit
        assert r["lds_limit"] == (min(163840 // r["lds_per_wg"], 1 << 20) if r["lds_per_wg"] > 0 else 1 << 20)
        assert r["wave_limit"] == 32 // r["waves_per_wg"]
        assert r["wg_per_cu"] == min(r["reg_limit"], r["lds_limit"], r["wave_limit"])
        # every compiled configuration fits one CDNA4 CU: LDS and workgroup size limits
        assert 0 <= r["lds_per_wg"] <= 163840, c["name"]
        assert c["threads"] <= 1024, c["name"]


def _kind(op):
    return {"gemm": nj.NNJIT_KIND_GEMM, "batched": nj.NNJIT_KIND_BATCHED, "gemv": nj.NNJIT_KIND_GEMV,
            "gemv_q4": nj.NNJIT_KIND_GEMV_Q4}[op.kind]


ALL_OPS = [(n, i) for n in workloads.WORKLOADS for i in range(len(workloads.workload(n)))]


@pytest.mark.parametrize("name,index", ALL_OPS)
def test_lite_space_is_dozens_and_ordered(lib, name, index):
    op = workloads.workload(name)[index]
    d = nj.mi355x_limits()
    dt = nj.NNJIT_F16 if op.dtype in ("f16", "q4") else nj.NNJIT_F32
    batch = op.group if op.kind == "gemv_q4" else op.batch   # a 4-bit GEMV is keyed by its group size
    ids, n, n_enum, n_naive = nj.nnjit_lite_space(_kind(op), dt, batch, op.M, op.N, op.K, d)
    assert 8 <= n <= 100, n            # "dozens", never empty
    assert n_naive > (10 * n if op.kind in ("gemm", "batched") else 2 * n)
    cfgs = nj.configs()
    fam = "gemv_q4" if op.kind == "gemv_q4" else ("gemv_" if op.kind == "gemv" else "gemm_") + op.dtype
    prev = {}
    for i in ids:
        c = cfgs[i]
        assert c["family"] == fam
        r = nj.nnjit_config_resources(i, d)
        assert c["threads"] <= d.max_threads_per_wg       # heuristic 5
        assert r["lds_per_wg"] <= d.lds_per_wg           # heuristic 6
        kind = c.get("direct", 0)                        # staging in registers / LDS direct copies
        if kind in prev:
            assert r["wg_per_cu"] <= prev[kind]          # evaluated from max to min Block_core, per kind
        prev[kind] = r["wg_per_cu"]
        if op.kind in ("gemm", "batched"):
            assert c["Mt"] <= max(16, 1 << (op.M - 1).bit_length())
    # deterministic
    assert nj.nnjit_lite_space(_kind(op), dt, batch, op.M, op.N, op.K, d)[0] == ids


def test_heuristic7_prefers_register_bound(lib):
    d = nj.mi355x_limits()
    ids, n, _, _ = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, 1024, 1024, 1024, d)
    cfgs = nj.configs()
    rs = [nj.nnjit_config_resources(i, d) for i in ids]
    # register-staged configurations are register bound; direct-copy ones,
    # whose staging lives in LDS, are LDS bound
    bound = [r["wg_per_cu"] == (r["lds_limit"] if cfgs[i]["direct"] else r["reg_limit"]) for i, r in zip(ids, rs)]
    assert all(bound) or n >= 8
    # both staging kinds are evaluated when both survive
    assert any(cfgs[i]["direct"] for i in ids) and any(not cfgs[i]["direct"] for i in ids)


def test_more_lds_never_shrinks_limits(lib):
    d = nj.mi355x_limits()
    d2 = nj.mi355x_limits()
    d2.lds_per_cu = 2 * d.lds_per_cu
    for c in nj.configs()[::7]:
        a = nj.nnjit_config_resources(c["id"], d)
        b = nj.nnjit_config_resources(c["id"], d2)
        assert b["lds_limit"] >= a["lds_limit"] and b["wg_per_cu"] >= a["wg_per_cu"]


def test_misaligned_shapes_get_element_load_configs(lib):
    d = nj.mi355x_limits()
    ids, n, _, _ = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, 100, 101, 99, d)
    cfgs = nj.configs()
    assert n >= 1 and all(cfgs[i]["vec"] == 4 for i in ids)
    ids, n, _, _ = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMM, nj.NNJIT_F32, 1, 100, 104, 96, d)
    assert all(cfgs[i]["vec"] == 16 for i in ids)


def test_microbench_groups_vary_one_primitive(lib):
    """The offline microbenchmark compares configurations that differ in
    exactly one primitive (besides derived fields); staging groups compare
    the two staging kinds on the same tile hierarchy, instruction shape and
    load width.  Every primitive, the new ones included (staging, LDS layout,
    unroll), has groups in the fp32 family."""
    from paper_2309_08978_amd.microbench import groups_for, PRIMITIVES, DERIVED, DIRECT_KEY
    cfgs = [c for c in nj.configs() if c["family"] == "gemm_f32"]
    per_prim = {}
    for prim in PRIMITIVES:
        per_prim[prim] = 0
        for grp in groups_for(cfgs, prim):
            per_prim[prim] += 1
            assert len(grp) >= 2
            members = [c for cs in grp.values() for c in cs]
            assert all(c[prim] == v for v, cs in grp.items() for c in cs)
            for c in members:
                assert c["split"] == 1
                if prim == "direct":
                    assert tuple(c[k] for k in DIRECT_KEY) == tuple(members[0][k] for k in DIRECT_KEY)
                else:
                    rest = {k: v for k, v in c.items() if k not in DERIVED and k != prim}
                    assert rest == {k: v for k, v in members[0].items() if k not in DERIVED and k != prim}
    for prim in ("direct", "layout", "unroll", "prefetch", "Kt", "vec"):
        assert per_prim[prim] >= 1, (prim, per_prim)


def test_consistent_table_is_generated_from_the_stored_measurement(lib):
    """csrc/consistent.inc is exactly what the microbenchmark's rule makes of
    the committed measurement, and no lite space of a workload shape holds a
    configuration with another setting of a primitive the table fixes."""
    from paper_2309_08978_amd import microbench as mb
    if os.path.exists(mb.MEASUREMENT):
        runs = json.load(open(mb.MEASUREMENT))["runs"]
        assert open(mb.TABLE).read() == mb.table_text(runs)
        fixed = mb.consistent_settings(runs)
    else:
        fixed = []
    cfgs = nj.configs()
    dev = nj.mi355x_limits()
    for name in workloads.WORKLOADS:
        for op in workloads.workload(name):
            if op.dtype not in ("f32", "f16") or op.M == 1:
                continue
            kind = nj.NNJIT_KIND_GEMM if op.batch == 1 else nj.NNJIT_KIND_BATCHED
            ids, _, _, _ = nj.nnjit_lite_space(kind, 1 if op.dtype == "f16" else 0, op.batch, op.M, op.N, op.K, dev)
            for i in ids:
                assert not mb.excluded_by(cfgs[i], fixed, cfgs), (name, op.name, cfgs[i]["name"])
    # the rule excludes something (when the table fixes anything)
    if fixed:
        assert any(mb.excluded_by(c, fixed, cfgs) for c in cfgs)


@pytest.mark.parametrize("N,K,G", [(4096, 4096, 128), (12288, 4096, 128), (4096, 11008, 128), (32000, 4096, 128),
                                   (4096, 4096, 32), (4096, 4096, 1), (4096, 300, 7), (5, 300, 64)])
def test_q4_lite_space(lib, N, K, G):
    """4-bit GEMV lite space: only its own family, never split; 16-byte
    configurations exactly when G % 32 == 0; K-slices and blocks in flight
    only where K has blocks for them (else the unfit fallback); evaluation
    order by workgroups per CU."""
    d = nj.mi355x_limits()
    ids, n, n_enum, n_naive = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMV_Q4, nj.NNJIT_F16, G, 1, N, K, d)
    assert 1 <= n <= 96 and n_naive > n
    cfgs = nj.configs()
    nblk = -(-K // 2048)
    fits = []
    prev = None
    for i in ids:
        c = cfgs[i]
        assert c["family"] == "gemv_q4" and c["split"] == 1
        assert (c["vec"] == 16) == (G % 32 == 0)
        fits.append(c["kslices"] <= nblk and (c["unroll"] == 1 or -(-nblk // c["kslices"]) >= c["unroll"]))
        r = nj.nnjit_config_resources(i, d)
        if prev is not None:
            assert r["wg_per_cu"] <= prev
        prev = r["wg_per_cu"]
    assert all(fits) or not any(fits)
    assert nj.nnjit_lite_space(nj.NNJIT_KIND_GEMV_Q4, nj.NNJIT_F16, G, 1, N, K, d)[0] == ids
    with pytest.raises(nj.NnjitError):
        nj.nnjit_lite_space(nj.NNJIT_KIND_GEMV_Q4, nj.NNJIT_F32, G, 1, N, K, d)


def _streamk_model(tiles, nslab, G):
    """The stream-K work split written out plainly (the GEMM kernel's segment
    loop and the fix-up kernel's contributor walk, as GemmParams documents
    them): returns (full tiles -> writer, partial slot writes, fix-up reads)."""
    units = tiles * nslab
    u0 = lambda w: w * units // G
    full, writes = {}, {}
    for w in range(G):
        su, end, first = u0(w), u0(w + 1), True
        while su < end:
            t = su // nslab
            ks = su - t * nslab
            ke = min(nslab, ks + (end - su))
            if ks == 0 and ke == nslab:
                assert t not in full
                full[t] = w
            else:
                slot = 2 * w + (0 if first else 1)
                assert slot not in writes, "a slot is written twice"
                writes[slot] = (t, ks, ke)
            su += ke - ks
            first = False
    reads = {}
    for b in range(1, G):
        ub = u0(b)
        t = ub // nslab
        tstart, tend = t * nslab, t * nslab + nslab
        if ub == tstart or u0(b - 1) > tstart:
            continue
        assert t not in reads, "two fix-up workgroups for one tile"
        w, slots = b - 1, []
        while w < G and u0(w) < tend:
            slots.append(2 * w + (0 if u0(w) >= tstart else 1))
            w += 1
        reads[t] = slots
    return full, writes, reads


@pytest.mark.parametrize("tiles,nslab,G", [(172, 256, 256), (192, 256, 256), (500, 256, 256), (64, 64, 256),
                                           (3, 5, 256), (1, 700, 256), (300, 7, 256), (256, 256, 256),
                                           (257, 100, 512), (40, 1024, 37)])
def test_streamk_split_covers_every_unit_once(tiles, nslab, G):
    """Every tile is either stored whole by one workgroup or summed by exactly
    one fix-up workgroup from partial slots that cover its K slabs exactly
    once, in K order; no slot is written twice and none lies outside the
    2 x G slots of the workspace."""
    G = min(G, tiles * nslab)
    full, writes, reads = _streamk_model(tiles, nslab, G)
    for t in range(tiles):
        assert (t in full) != (t in reads), t
        if t in reads:
            pieces = [writes[s] for s in reads[t]]
            assert all(p[0] == t for p in pieces)
            ranges = [(p[1], p[2]) for p in pieces]
            assert ranges[0][0] == 0 and ranges[-1][1] == nslab
            assert all(a[1] == b[0] for a, b in zip(ranges, ranges[1:])), "pieces out of K order or overlapping"
            assert len(reads[t]) >= 2
    assert sorted(s for ss in reads.values() for s in ss) == sorted(writes)
    assert all(0 <= s < 2 * G for s in writes)
