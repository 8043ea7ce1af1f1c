"""GPU parity of the 4-bit weight-only GEMV (nnjit_gemv_q4) against the CPU
oracle, through the C-ABI.

* every configuration id of the family, forced, on exact-arithmetic inputs
  (x in {-8..8}, power-of-two scales varying by output and group) at ragged
  shapes: an output count that ends inside a workgroup, a K that ends inside
  a word, a chunk and a 2048-input block, padding words holding random codes
  -- bit-exact, and identical when run twice;
* edge cases: odd and unit group sizes, a group larger than K, K = 0
  (zeros), N = 0 (no-op), K = 1, padded leading dimensions, misaligned
  operands (word-load fallback);
* the Llama-2-7B decode shapes at full size, tuned, on the workload's own
  value recipe: the fp32 bar (rel-Frobenius 1e-5 and |err| <= 2e-6 K
  max|x| max|W| per element, max|W| <= 8 max|s|) on every output;
* tuned dispatch equals the forced configuration; graph replays equal eager.
"""
import numpy as np
import pytest

import oracle
from oracle import accept
import paper_2309_08978_amd as nj
import workloads
from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu


def _run(x, Wq, S, group, N, cfg=None, pad=0):
    """y on the GPU; ``pad`` > 0 offsets every operand by that many elements
    inside a larger buffer (misaligned base pointers)."""
    import torch
    if pad:
        bx = torch.zeros(x.size + pad, dtype=torch.float16, device="cuda:0")
        bw = torch.zeros(Wq.size + pad, dtype=torch.int32, device="cuda:0")
        bs = torch.zeros(S.size + pad, dtype=torch.float16, device="cuda:0")
        bx[pad:] = dev(x)
        bw[pad:] = dev(Wq.view(np.int32).reshape(-1))
        bs[pad:] = dev(S.reshape(-1))
        dx, dW, dS = bx[pad:], bw[pad:].view(Wq.shape), bs[pad:].view(S.shape)
    else:
        dx, dW, dS = dev(x), dev(Wq.view(np.int32)), dev(S)
    return host(nj.gemv_q4(dx, dW, dS, group, N, cfg=cfg))


def _bound_inputs(x, S):
    # max|W| <= 8 max|s| (|q - 8| <= 8): the per-element fp32 bound uses it
    smax = float(np.max(np.abs(S.astype(np.float64)))) if S.size else 0.0
    return x.astype(np.float64)[None, :], np.array([[8.0 * smax]])


@pytest.fixture(scope="module")
def q4_configs():
    nj.load()
    return [c for c in nj.configs() if c["family"] == "gemv_q4"]


def test_every_config_bit_exact(q4_configs):
    N = 1037
    n_run = 0
    # 16-byte configurations: G a multiple of 32, rows padded to a multiple of 4
    # words; word configurations: any G, unpadded rows
    for vec, K, G, ldq in ((True, 4201, 64, 528), (False, 4201, 48, None)):
        x, Wq, S = workloads.q4_operands(7, K, N, G, ldq=ldq, recipe="q4_int")
        R = oracle.gemv_q4(x, Wq, S, G, N)
        for c in q4_configs:
            if (c["vec"] == 16) != vec:
                continue
            print(f"cfg {c['id']} {c['name']} N={N} K={K} G={G}", flush=True)
            y1 = _run(x, Wq, S, G, N, cfg=c["id"])
            y2 = _run(x, Wq, S, G, N, cfg=c["id"])
            assert np.array_equal(y1, R), (c["name"], np.flatnonzero(y1 != R)[:10])
            assert np.array_equal(y1, y2)
            n_run += 1
    assert n_run == len(q4_configs)


@pytest.mark.parametrize("N,K,G,ldq", [(1037, 300, 7, None), (1037, 300, 1, None), (1037, 300, 1024, 40),
                                       (1037, 1, 128, 4), (64, 4096, 128, None), (8, 77, 32, None),
                                       (13, 130, 32, 20), (1, 33, 2, None), (4128, 2048, 64, None),
                                       (300, 8192, 128, None), (700, 6200, 96, 776)])
def test_edge_shapes_bit_exact(N, K, G, ldq):
    print(f"N={N} K={K} G={G} ldq={ldq}", flush=True)
    x, Wq, S = workloads.q4_operands(N * 7 + K, K, N, G, ldq=ldq, recipe="q4_int")
    R = oracle.gemv_q4(x, Wq, S, G, N)
    assert np.array_equal(_run(x, Wq, S, G, N), R)


def test_k_zero_writes_zeros_and_n_zero_is_noop():
    import torch
    y = torch.full((96,), 7.0, dtype=torch.float32, device="cuda:0")
    nj.check(nj.nnjit_gemv_q4(96, 0, 128, None, None, 0, None, 0, y, None))
    assert np.array_equal(host(y), np.zeros(96))
    assert nj.nnjit_gemv_q4(0, 64, 32, None, None, 8, None, 2, None, None) == nj.NNJIT_OK


def test_padded_leading_dimensions():
    N, K, G = 1037, 4200, 64
    x, Wq, S = workloads.q4_operands(11, K, N, G, ldq=K // 8 + 7 * 4, lds=K // G + 9, recipe="q4_int")
    R = oracle.gemv_q4(x, Wq, S, G, N)
    assert np.array_equal(_run(x, Wq, S, G, N), R)
    # a row length that breaks the 16-byte conditions: the word-load configuration runs
    x, Wq, S = workloads.q4_operands(12, K, N, G, ldq=K // 8 + 1, lds=K // G + 3, recipe="q4_int")
    R = oracle.gemv_q4(x, Wq, S, G, N)
    assert np.array_equal(_run(x, Wq, S, G, N), R)


@pytest.mark.parametrize("pad", [1, 3])
def test_misaligned_operands_use_fallback(pad):
    N, K, G = 1037, 4200, 64
    x, Wq, S = workloads.q4_operands(13, K, N, G, recipe="q4_int")
    R = oracle.gemv_q4(x, Wq, S, G, N)
    assert np.array_equal(_run(x, Wq, S, G, N, pad=pad), R)
    vec = next(c["id"] for c in nj.configs() if c["family"] == "gemv_q4" and c["vec"] == 16)
    import torch
    buf = torch.zeros(Wq.size + 1, dtype=torch.int32, device="cuda:0")
    y = torch.empty(N, dtype=torch.float32, device="cuda:0")
    rc = nj.nnjit_gemv_q4_config(vec, N, K, G, dev(x), buf[1:], K // 8, dev(S), K // G, y, None)
    assert rc == nj.NNJIT_EINVAL


Q4_OPS = list(range(len(workloads.workload("llama2_7b_decode_q4"))))


@pytest.mark.parametrize("index", Q4_OPS, ids=[op.name for op in workloads.workload("llama2_7b_decode_q4")])
def test_llama_decode_q4_parity(index):
    import torch
    name = "llama2_7b_decode_q4"
    op = workloads.workload(name)[index]
    x, Wq, S = workloads.op_inputs(name, index)
    cfg = nj.check(nj.nnjit_tune_gemv_q4(op.N, op.K, op.group))
    st = nj.nnjit_last_tune_stats_ex()
    print(f"{op.name}: tuned -> {nj.nnjit_config_info(cfg)} | {st['best_us']:.2f} us, lite {st['n_lite']}, "
          f"timed {st['n_timed']}, tune {st['wall_ms']:.0f} ms", flush=True)
    lite, _, _, _ = nj.nnjit_lite_space(nj.NNJIT_KIND_GEMV_Q4, nj.NNJIT_F16, op.group, 1, op.N, op.K)
    assert cfg in lite
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMV_Q4, nj.NNJIT_F16, op.group, 1, op.N, op.K) == cfg
    y = _run(x, Wq, S, op.group, op.N)
    assert np.array_equal(y, _run(x, Wq, S, op.group, op.N, cfg=cfg))
    R = oracle.gemv_q4(x, Wq, S, op.group, op.N)
    A, B = _bound_inputs(x, S)
    res = accept.check(y[None, :], R[None, :], A, B, "f32", K=op.K)
    print(f"   rel_fro={res['rel_fro']:.3e} max_err={res['max_err']:.3e} bound={res['elt_bound']:.3e}", flush=True)
    assert res["ok"], res
    torch.cuda.empty_cache()


def test_graph_replay_matches_eager():
    """A tuned, split 4-bit GEMV captured in a graph: every replay, with
    eager work between replays, equals the eager result bit for bit."""
    import torch
    name = "llama2_7b_decode_q4"
    op = workloads.workload(name)[1]
    x, Wq, S = workloads.op_inputs(name, 1)
    nj.check(nj.nnjit_tune_gemv_q4(op.N, op.K, op.group))
    dx, dW, dS = dev(x), dev(Wq.view(np.int32)), dev(S)
    eager = host(nj.gemv_q4(dx, dW, dS, op.group, op.N))
    side = torch.cuda.Stream()
    y = torch.empty(op.N, dtype=torch.float32, device="cuda:0")
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        nj.gemv_q4(dx, dW, dS, op.group, op.N, y=y, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        nj.gemv_q4(dx, dW, dS, op.group, op.N, y=y, stream=side)
    for _ in range(3):
        y.fill_(-1.0)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host(y), eager)
        other = host(nj.gemv_q4(dx, dW, dS, op.group, op.N))   # eager work between replays
        assert np.array_equal(other, eager)


def test_kernel_database_round_trip(tmp_path):
    op = workloads.workload("llama2_7b_decode_q4")[1]
    nj.nnjit_cache_clear()
    cfg = nj.check(nj.nnjit_tune_gemv_q4(op.N, op.K, op.group))
    path = str(tmp_path / "db.txt")
    assert nj.check(nj.nnjit_cache_save(path)) >= 1
    nj.nnjit_cache_clear()
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMV_Q4, nj.NNJIT_F16, op.group, 1, op.N, op.K) == nj.NNJIT_ENOCFG
    assert nj.check(nj.nnjit_cache_load(path)) >= 1
    assert nj.nnjit_cached_config(nj.NNJIT_KIND_GEMV_Q4, nj.NNJIT_F16, op.group, 1, op.N, op.K) == cfg
    nj.nnjit_cache_clear()
