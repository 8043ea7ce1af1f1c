"""GPU pins fixed by closed forms rather than by the oracle, plus brute force
over tiny shapes.

* identity and permutation operands (real-valued, seeded): every output is a
  single product a * 1 plus exact zeros, so every configuration of every
  family (split-K included) must reproduce the operand bit for bit;
* rank-1 operands with integer entries: C[i][j] = K u_i z_j and
  C[i][j] = K (K - 1) / 2 (all partial sums are integers below 2^24, exact in
  fp32 in any order), on every configuration and on long K with the tuned
  configuration;
* every shape (M, N, K) in {1..8}^3 and in {1, 17, 63, 129, 257}^3, both
  dtypes, default configuration, against the oracle within the acceptance
  bounds.
"""
import itertools

import numpy as np
import pytest

import oracle
from oracle import accept
import paper_2309_08978_amd as nj
import workloads
from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu

FAMILY_DTYPE = {"gemm_f32": "f32", "gemm_f16": "f16", "gemv_f32": "f32", "gemv_f16": "f16"}
NP = {"f32": np.float32, "f16": np.float16}


def _shapes(family, vec):
    """(M, N, K) with K <= N (a permutation of the K rows into N columns);
    vector configurations need N and K multiples of 8."""
    if family.startswith("gemv"):
        return (1, 1032, 997) if vec else (1, 1027, 997)
    return (291, 264, 200) if vec else (291, 259, 197)


def _run(cfg_id, A, B):
    import torch
    dA, dB = dev(A), dev(B)
    C = torch.full((A.shape[0], B.shape[1]), float("nan"), dtype=torch.float32, device="cuda:0")
    nj.matmul(dA, dB, C, cfg=cfg_id)
    return host(C)


def _permutation(K, N, seed):
    rng = np.random.default_rng(seed)
    cols = rng.permutation(N)[:K]
    P = np.zeros((K, N))
    P[np.arange(K), cols] = 1.0
    return P, cols


@pytest.mark.parametrize("family", ["gemm_f32", "gemm_f16", "gemv_f32", "gemv_f16"])
def test_permutation_and_identity_every_config(family):
    dt = FAMILY_DTYPE[family]
    t = NP[dt]
    n = 0
    for c in nj.configs():
        if c["family"] != family:
            continue
        M, N, K = _shapes(family, c["vec"] == 16)
        A, _ = workloads.random_operands(700 + n % 7, 1, M, K, N, dt)
        P, cols = _permutation(K, N, 800 + n % 5)
        C = _run(c["id"], A, P.astype(t))
        expect = np.zeros((M, N))
        expect[:, cols] = A.astype(np.float64)
        assert np.array_equal(C, expect), f"permutation: config {c['id']} {c['name']} split={c['split']}"
        if family.startswith("gemm"):
            # A = I (K x K): C = B
            _, B = workloads.random_operands(900 + n % 3, 1, K, K, N, dt)
            C = _run(c["id"], np.eye(K).astype(t), B)
            assert np.array_equal(C, B.astype(np.float64)), f"identity: config {c['id']} {c['name']}"
        n += 1
    assert n > 0


@pytest.mark.parametrize("family", ["gemm_f32", "gemm_f16", "gemv_f32", "gemv_f16"])
def test_rank_one_closed_forms_every_config(family):
    dt = FAMILY_DTYPE[family]
    t = NP[dt]
    n = 0
    for c in nj.configs():
        if c["family"] != family:
            continue
        M, N, K = _shapes(family, c["vec"] == 16)
        u = (np.arange(M) % 7) - 3.0
        z = (np.arange(N) % 5) - 2.0
        # (a) A[i][k] = u_i, B[k][j] = z_j  ->  C = K u_i z_j
        C = _run(c["id"], np.repeat(u[:, None], K, 1).astype(t), np.repeat(z[None, :], K, 0).astype(t))
        assert np.array_equal(C, K * np.outer(u, z)), f"rank-1 (a): config {c['id']} {c['name']}"
        # (c) A[i][k] = k, B = 1  ->  C = K (K - 1) / 2
        C = _run(c["id"], np.tile(np.arange(K, dtype=np.float64), (M, 1)).astype(t), np.ones((K, N), dtype=t))
        assert np.all(C == K * (K - 1) / 2), f"rank-1 (c): config {c['id']} {c['name']}"
        n += 1
    assert n > 0


@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("M,N,K", [(1, 4096, 5792), (128, 768, 5792), (512, 520, 2048)])
def test_rank_one_long_k_tuned(dt, M, N, K):
    """Long K through the tuned configuration (split-K where the tuner picks
    it): C = K (K - 1) / 2 exactly (K <= 5793 keeps every sum below 2^24;
    fp16 holds the integers up to 2048 exactly, so its k runs modulo 2048)."""
    t = NP[dt]
    code = nj.NNJIT_F16 if dt == "f16" else nj.NNJIT_F32
    nj.check(nj.nnjit_tune(M, N, K, code))
    k = np.arange(K, dtype=np.float64)
    if dt == "f16":
        k = k % 2048
    A = np.tile(k, (M, 1)).astype(t)
    C = _run(None, A, np.ones((K, N), dtype=t))
    assert np.all(C == k.sum())


def _tiny_shapes():
    small = list(itertools.product(range(1, 9), repeat=3))
    ragged = list(itertools.product([1, 17, 63, 129, 257], repeat=3))
    return small + ragged


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_tiny_and_ragged_shapes_default_config(dt):
    bad = []
    for s, (M, N, K) in enumerate(_tiny_shapes()):
        A, B = workloads.random_operands(5000 + s, 1, M, K, N, dt)
        C = _run(None, A, B)
        res = accept.check(C, oracle.matmul(A, B), A, B, dt)
        if not res["ok"]:
            bad.append(((M, N, K), res))
    assert not bad, f"{len(bad)} shapes fail, first: {bad[:3]}"
