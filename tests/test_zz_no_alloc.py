"""The allocation-free entry point (nnjit_batched_matmul_noalloc) through the
C-ABI: on the same operands it gives the same result as
nnjit_batched_matmul -- the same configuration, its split-K partials in the
library's fixed scratch instead of a per-stream buffer -- on two calls in a
row, the second with a smaller input; a configuration whose partials exceed
the fixed scratch is refused before any launch."""
import numpy as np
import pytest

import oracle
import paper_2309_08978_amd as nj
import workloads
from tests.gpu_util import dev, host, dtype_code

pytestmark = pytest.mark.gpu


def _noalloc(dA, dB, C, dt, stream=None):
    b, M, K = dA.shape
    N = dB.shape[2]
    return nj.nnjit_batched_matmul_noalloc(b, M, N, K, dA, K, M * K, dB, N, K * N, C, N, M * N, dt, stream)


def _reference(dA, dB, dt):
    import torch
    b, M, K = dA.shape
    N = dB.shape[2]
    C = torch.full((b, M, N), float("nan"), dtype=torch.float32, device="cuda:0")
    nj.check(nj.nnjit_batched_matmul(b, M, N, K, dA, K, M * K, dB, N, K * N, C, N, M * N, dt, None))
    return host(C)


def _pair(dt, big, small, seed, force=None, monkeypatch=None):
    """Two no-alloc calls in a row (big, then small) against the allocating
    entry point; small-integer operands, so both must equal the oracle
    exactly as well."""
    import torch
    outs = []
    for i, (b, M, N, K) in enumerate((big, small)):
        A, B = workloads.small_int_operands(seed + i, b, M, K, N, dt)
        A3, B3 = A.reshape(b, M, K), B.reshape(b, K, N)
        dA, dB = dev(A3), dev(B3)
        code = dtype_code(dt)
        C = torch.full((b, M, N), float("nan"), dtype=torch.float32, device="cuda:0")
        rc = _noalloc(dA, dB, C, code)
        assert rc == nj.NNJIT_OK, nj.nnjit_last_error()
        got = host(C)
        assert np.array_equal(got, _reference(dA, dB, code)), f"{dt} {b}x{M}x{N}x{K}"
        assert np.array_equal(got, oracle.matmul(A3, B3)), f"{dt} {b}x{M}x{N}x{K} vs oracle"
        outs.append(got)
    return outs


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_noalloc_matches_allocating_entry_point_split_k(all_split_configs, dt, monkeypatch):
    """A forced split-K configuration (its partials in the fixed scratch),
    then a smaller product on the same scratch: both equal the allocating
    entry point's result and the oracle's."""
    cfg = all_split_configs[dt]
    monkeypatch.setenv("NNJIT_FORCE_CONFIG", str(cfg))
    nj.nnjit_cache_clear()   # the library reads its environment here
    try:
        _pair(dt, (3, 200, 264, 1024), (1, 70, 136, 512), 7100 + (dt == "f16"))
    finally:
        monkeypatch.delenv("NNJIT_FORCE_CONFIG")
        nj.nnjit_cache_clear()


@pytest.mark.parametrize("name,index", [("bart_base_layer_seq128_f32", 3), ("llama2_7b_decode_f16", 1),
                                        ("llama2_7b_decode_f32", 4), ("t5_large_layer_b4s256_f32", 7)])
def test_noalloc_tuned_workload_shapes(name, index):
    """Tuned workload shapes (split-K GEMM and GEMV among them), then a
    smaller product: the no-alloc call equals the allocating one."""
    op = workloads.workload(name)[index]
    code = dtype_code(op.dtype)
    if op.batch == 1:
        nj.check(nj.nnjit_tune(op.M, op.N, op.K, code))
    else:
        nj.check(nj.nnjit_tune_batched(op.batch, op.M, op.N, op.K, code))
    big = (op.batch, op.M, op.N, op.K)
    small = (1, max(1, op.M // 2), max(8, op.N // 4 // 8 * 8), max(8, op.K // 2 // 8 * 8))
    _pair(op.dtype, big, small, 7300 + index)


def test_noalloc_refuses_oversized_scratch(monkeypatch):
    """Split 16 of a 2048 x 2048 output needs 256 MiB of partials, above the
    128 MiB fixed scratch: refused with NNJIT_ENOMEM, C untouched."""
    import torch
    cfg = next(c for c in nj.configs() if c["family"] == "gemm_f32" and c["vec"] == 16 and c["split"] == 16)
    monkeypatch.setenv("NNJIT_FORCE_CONFIG", str(cfg["id"]))
    nj.nnjit_cache_clear()
    try:
        M = N = 2048
        K = 1024
        dA = torch.ones((1, M, K), dtype=torch.float32, device="cuda:0")
        dB = torch.ones((1, K, N), dtype=torch.float32, device="cuda:0")
        C = torch.full((1, M, N), 7.0, dtype=torch.float32, device="cuda:0")
        rc = _noalloc(dA, dB, C, nj.NNJIT_F32)
        assert rc == nj.NNJIT_ENOMEM, rc
        assert "fixed scratch" in nj.nnjit_last_error()
        assert bool((C == 7.0).all())
    finally:
        monkeypatch.delenv("NNJIT_FORCE_CONFIG")
        nj.nnjit_cache_clear()


@pytest.fixture(scope="module")
def all_split_configs():
    nj.load()
    cf = nj.configs()
    return {"f32": next(c["id"] for c in cf if c["family"] == "gemm_f32" and c["vec"] == 16 and c["split"] == 4),
            "f16": next(c["id"] for c in cf if c["family"] == "gemm_f16" and c["vec"] == 16 and c["split"] == 4)}


def test_noalloc_captured_in_a_graph(all_split_configs, monkeypatch):
    """The use the entry point exists for: calls recorded into a HIP graph on a
    stream no call has used before (no scratch of its own) -- a split-K
    configuration, whose partials go to the fixed scratch -- replay correctly
    several times, with eager work between the replays, every replay equal
    to the eager result and to the oracle."""
    import torch
    cfg = all_split_configs["f32"]
    monkeypatch.setenv("NNJIT_FORCE_CONFIG", str(cfg))
    nj.nnjit_cache_clear()   # the library reads its environment here
    try:
        M, N, K = 96, 200, 520
        A, B = workloads.small_int_operands(7400, 1, M, K, N, "f32")
        R = oracle.matmul(A, B)
        dA, dB = dev(A.reshape(1, M, K)), dev(B.reshape(1, K, N))
        eager = torch.full((1, M, N), float("nan"), dtype=torch.float32, device="cuda:0")
        assert _noalloc(dA, dB, eager, nj.NNJIT_F32) == nj.NNJIT_OK, nj.nnjit_last_error()
        torch.cuda.synchronize()
        assert np.array_equal(host(eager)[0], R)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            C = torch.full((1, M, N), float("nan"), dtype=torch.float32, device="cuda:0")
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            rc = _noalloc(dA, dB, C, nj.NNJIT_F32, side)
        assert rc == nj.NNJIT_OK, nj.nnjit_last_error()
        other = torch.full((1, M, N), float("nan"), dtype=torch.float32, device="cuda:0")
        for rep in range(4):
            C.fill_(float("nan"))
            assert _noalloc(dA, dB, other, nj.NNJIT_F32) == nj.NNJIT_OK   # eager use of the same scratch
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            assert np.array_equal(host(C)[0], R), f"replay {rep}"
            assert np.array_equal(host(other)[0], R)
    finally:
        monkeypatch.delenv("NNJIT_FORCE_CONFIG")
        nj.nnjit_cache_clear()
