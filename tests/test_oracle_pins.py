"""Pins of the CPU oracle to things other than itself (CPU only).

The oracle evaluates R = A . B (the MatMul / BatchMatMul of the paper's
kernel table, Table 3) in fp64.  Each test below ties it to a fact the
mathematics fixes:

* hand-worked examples (tests/golden/matmul_hand_examples.json);
* identity and permutation operands: the result is a copy of an operand;
* rank-1 operands with closed-form sums;
* small integers, checked against exact int64 arithmetic;
* tiny shapes, checked against exact rational arithmetic within the fp64
  summation error bound;
* numpy's float64 product (a different library routine);
* thread-count independence (fixed per-element order);
* the binary16 decoder against numpy over all 65536 bit patterns.

``test_planted_mistakes_are_caught`` compiles copies of oracle.c with a
mistake planted in them (a dropped term, a wrong sign, a wrong index, a
transposed operand, a wrong fp16 exponent bias) and checks that the pins
reject every one.
"""
import json
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import accept
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "matmul_hand_examples.json")


# ----------------------------------------------------------------- pin suite
# Each pin takes an Oracle instance and raises AssertionError on failure, so
# the same suite runs on the real oracle and on planted-mistake builds.

def pin_golden(o):
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        if c["dtype"] == "f16":
            A = np.array(c["A_bits"], dtype=np.uint16).view(np.float16)
            B = np.array(c["B_bits"], dtype=np.uint16).view(np.float16)
        else:
            A = np.array(c["A"], dtype=np.float32)
            B = np.array(c["B"], dtype=np.float32)
        R = o.matmul(A, B)
        assert np.array_equal(R, np.array(c["C"], dtype=np.float64)), c["name"]


def pin_identity(o):
    rng = np.random.default_rng(11)
    for dt in (np.float32, np.float16):
        A = rng.standard_normal((37, 29)).astype(dt)
        I29 = np.eye(29, dtype=dt)
        I37 = np.eye(37, dtype=dt)
        assert np.array_equal(o.matmul(A, I29), A.astype(np.float64)), "A.I == A"
        assert np.array_equal(o.matmul(I37, A), A.astype(np.float64)), "I.A == A"
        x = np.zeros((1, 29), dtype=dt)
        x[0, 5] = 1
        W = rng.standard_normal((29, 41)).astype(dt)
        assert np.array_equal(o.matmul(x, W)[0], W[5].astype(np.float64)), "e_k.W == W[k]"


def pin_permutation(o):
    rng = np.random.default_rng(12)
    K = 23
    perm = rng.permutation(K)
    P = np.zeros((K, K), dtype=np.float32)
    P[np.arange(K), perm] = 1.0
    A = rng.standard_normal((19, K)).astype(np.float32)
    R = o.matmul(A, P)
    assert np.array_equal(R[:, perm], A.astype(np.float64)), "column permutation"


def pin_rank1(o):
    for (M, K, N) in [(9, 40, 7), (5, 301, 11), (3, 1, 4)]:
        i = np.arange(M)
        j = np.arange(N)
        k = np.arange(K)
        u = (i % 7 - 3).astype(np.float64)
        z = (j % 5 - 2).astype(np.float64)
        v = (k % 3 - 1).astype(np.float64)
        # (a) A[i,k] = u_i, B[k,j] = z_j  ->  C = K u_i z_j
        A = np.repeat(u[:, None], K, axis=1).astype(np.float32)
        B = np.repeat(z[None, :], K, axis=0).astype(np.float32)
        assert np.array_equal(o.matmul(A, B), K * np.outer(u, z)), "rank-1 (a)"
        # (b) A[i,k] = u_i v_k, B[k,j] = v_k z_j  ->  C = u_i z_j * sum_k v_k^2
        #     v_k^2 is 1 unless k = 1 mod 3, so sum = K - #{k < K : k = 1 mod 3}
        A = np.outer(u, v).astype(np.float32)
        B = np.outer(v, z).astype(np.float32)
        n1 = (K + 1) // 3
        assert np.array_equal(o.matmul(A, B), (K - n1) * np.outer(u, z)), "rank-1 (b)"
        # (c) A[i,k] = k, B = 1  ->  C = K (K - 1) / 2
        A = np.repeat(k[None, :].astype(np.float32), M, axis=0)
        B = np.ones((K, N), dtype=np.float32)
        assert np.all(o.matmul(A, B) == K * (K - 1) / 2), "rank-1 (c)"


def pin_small_integers(o):
    for seed, (b, M, K, N) in enumerate([(1, 33, 65, 17), (3, 8, 129, 5), (1, 1, 257, 63)]):
        for dt in ("f32", "f16"):
            A, B = workloads.small_int_operands(seed, b, M, K, N, dt)
            exact = np.matmul(A.astype(np.int64), B.astype(np.int64))
            R = o.matmul(A, B)
            assert np.array_equal(R, exact.astype(np.float64)), f"int {dt} {(b, M, K, N)}"


def _gamma(n):
    u = 2.0 ** -53
    return n * u / (1 - n * u)


def pin_rational_bruteforce(o):
    rng = np.random.default_rng(13)
    shapes = [(m, n, k) for m in (1, 2, 3) for n in (1, 2, 5) for k in (1, 2, 3, 8)]
    shapes += [(2, 3, 17), (1, 4, 33), (3, 1, 65)]
    for (M, N, K) in shapes:
        A = rng.standard_normal((M, K)).astype(np.float32)
        B = rng.standard_normal((K, N)).astype(np.float32)
        R = o.matmul(A, B)
        Af = [[Fraction(float(x)) for x in row] for row in A]
        Bf = [[Fraction(float(x)) for x in row] for row in B]
        for i in range(M):
            for j in range(N):
                exact = sum((Af[i][k] * Bf[k][j] for k in range(K)), Fraction(0))
                absum = sum(abs(Af[i][k] * Bf[k][j]) for k in range(K))
                bound = _gamma(max(K - 1, 1)) * float(absum)
                assert abs(Fraction(R[i, j]) - exact) <= Fraction(bound), (M, N, K, i, j)


def pin_numpy_f64(o):
    for seed, (b, M, K, N) in enumerate([(1, 64, 768, 96), (4, 17, 33, 65), (1, 1, 1000, 300)]):
        A, B = workloads.random_operands(100 + seed, b, M, K, N, "f32")
        R = o.matmul(A, B)
        ref = np.matmul(A.astype(np.float64), B.astype(np.float64))
        den = np.abs(A.astype(np.float64)) @ np.abs(B.astype(np.float64))
        assert np.all(np.abs(R - ref) <= 4 * K * 2.0 ** -53 * den), (b, M, K, N)


def pin_f16_decode(o):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = o.f16_to_f64(bits)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def _q4_pack(codes):
    """uint32 words [N, ceil(K / 8)] from integer codes [N, K]: input k of row n
    in bits 4 (k % 8) .. of word k / 8 -- written independently of the oracle."""
    codes = np.asarray(codes, dtype=np.uint32)
    N, K = codes.shape
    words = np.zeros((N, (K + 7) // 8), dtype=np.uint32)
    for k in range(K):
        words[:, k // 8] |= codes[:, k] << np.uint32(4 * (k % 8))
    return words


def pin_q4_golden(o):
    """Hand-worked 4-bit example (tests/golden/gemv_q4_hand.json)."""
    with open(os.path.join(os.path.dirname(GOLDEN), "gemv_q4_hand.json")) as f:
        g = json.load(f)
    y = o.gemv_q4(np.array(g["x"], dtype=np.float16), np.array(g["words"], dtype=np.uint32),
                  np.array(g["scales"], dtype=np.float16), g["G"], g["N"])
    assert np.array_equal(y, np.array(g["y"]))


def pin_q4_zero_code(o):
    """Every code 8 encodes weight 0: y = 0 exactly for any x and scales."""
    rng = np.random.default_rng(31)
    N, K, G = 24, 37, 8
    x = rng.standard_normal(K).astype(np.float16)
    S = rng.standard_normal((N, (K + G - 1) // G)).astype(np.float16)
    y = o.gemv_q4(x, _q4_pack(np.full((N, K), 8)), S, G, N)
    assert np.array_equal(y, np.zeros(N))


def pin_q4_one_hot(o):
    """A single non-zero weight: y[n0] = x[k0] (q - 8) s[n0][k0 / G], exact;
    every other output 0."""
    N, K, G = 16, 20, 6
    rng = np.random.default_rng(32)
    x = rng.standard_normal(K).astype(np.float16)
    S = rng.standard_normal((N, (K + G - 1) // G)).astype(np.float16)
    for k0, n0, q in [(0, 0, 15), (13, 9, 0), (19, 15, 3)]:
        codes = np.full((N, K), 8)
        codes[n0, k0] = q
        y = o.gemv_q4(x, _q4_pack(codes), S, G, N)
        want = np.zeros(N)
        want[n0] = float(x[k0]) * (q - 8) * float(S[n0, k0 // G])
        assert np.array_equal(y, want), (k0, n0, q)


def pin_q4_integers(o):
    """Integer x and unit scales: the exact int64 product of (q - 8) and x."""
    rng = np.random.default_rng(33)
    N, K, G = 40, 130, 32
    x = rng.integers(-8, 9, K)
    codes = rng.integers(0, 16, (N, K))
    y = o.gemv_q4(x.astype(np.float16), _q4_pack(codes), np.ones((N, (K + G - 1) // G), np.float16), G, N)
    assert np.array_equal(y, ((codes.astype(np.int64) - 8) @ x.astype(np.int64)).astype(np.float64))


def pin_q4_numpy(o):
    """Random codes and scales vs numpy: unpack, dequantise, float64 matmul."""
    rng = np.random.default_rng(34)
    N, K, G = 64, 300, 128
    x = rng.standard_normal(K).astype(np.float16)
    codes = rng.integers(0, 16, (N, K))
    S = (rng.standard_normal((N, (K + G - 1) // G)) * 0.01).astype(np.float16)
    W = ((codes - 8).astype(np.float64) * S.astype(np.float64)[:, np.arange(K) // G]).T   # W[k][n]
    ref = x.astype(np.float64) @ W
    y = o.gemv_q4(x, _q4_pack(codes), S, G, N)
    bound = 1e-13 * (np.abs(x.astype(np.float64)) @ np.abs(W))
    assert np.all(np.abs(y - ref) <= bound)


PINS = [pin_golden, pin_identity, pin_permutation, pin_rank1, pin_small_integers,
        pin_rational_bruteforce, pin_numpy_f64, pin_f16_decode,
        pin_q4_golden, pin_q4_zero_code, pin_q4_one_hot, pin_q4_integers, pin_q4_numpy]


@pytest.fixture(scope="module")
def real():
    return oracle.default()


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(real, pin):
    pin(real)


def test_thread_count_independent(real):
    A, B = workloads.random_operands(7, 2, 45, 513, 1030, "f32")
    r1 = real.matmul(A, B, nthreads=1)
    rn = real.matmul(A, B, nthreads=max(2, real.max_threads()))
    assert np.array_equal(r1, rn)


def test_degenerate_shapes(real):
    A = np.zeros((4, 0), dtype=np.float32)
    B = np.zeros((0, 5), dtype=np.float32)
    assert np.array_equal(real.matmul(A, B), np.zeros((4, 5)))
    assert real.matmul(np.zeros((0, 3), np.float32), np.ones((3, 2), np.float32)).shape == (0, 2)


# ------------------------------------------------------------- the checker

def test_checker_rejects_just_beyond_bound():
    A, B = workloads.random_operands(21, 1, 64, 256, 96, "f32")
    R = oracle.matmul(A, B)
    res = accept.check(R.astype(np.float32), R, A, B, "f32")
    assert res["ok"]
    bound = res["elt_bound"]
    C = R.copy()
    C[3, 5] += 0.99 * bound
    assert accept.check(C, R, A, B, "f32")["ok"]
    C[3, 5] += 0.02 * bound
    assert not accept.check(C, R, A, B, "f32")["ok"]
    C = R.copy()
    C[0, 0] = np.nan
    assert not accept.check(C, R, A, B, "f32")["ok"]
    C = R.copy() * (1 + 3e-3)
    assert not accept.check(C, R, A, B, "f16")["ok"]
    assert accept.check(R * (1 + 1e-3), R, A, B, "f16")["ok"]
    Z = np.zeros((2, 2))
    assert accept.check(Z, Z, np.zeros((2, 3)), np.zeros((3, 2)), "f32")["ok"]
    Z2 = Z.copy()
    Z2[1, 1] = 1e-30
    assert not accept.check(Z2, Z, np.zeros((2, 3)), np.zeros((3, 2)), "f32")["ok"]


# --------------------------------------------------------- planted mistakes

MUTANTS = {
    "dropped_last_term": ("for (int64_t k = 0; k < K; ++k) {\n            const double a",
                          "for (int64_t k = 0; k < K - 1; ++k) {\n            const double a"),
    "wrong_sign": ("r[j] += a * brow[j]", "r[j] -= a * brow[j]"),
    "wrong_b_index": ("const double *brow = Bd + b * strideB + k * ldb;",
                      "const double *brow = Bd + b * strideB + ((k + 1) % K) * ldb;"),
    "transposed_a": ("Ad[b * strideA + i * lda + k]",
                     "Ad[b * strideA + (k % M) * lda + (i % K)]"),
    "f16_bias_off_by_one": ("int p = e - 15;", "int p = e - 14;"),
    "f16_subnormal_scale": ("(double)f / 1024.0 / 16384.0", "(double)f / 1024.0 / 32768.0"),
    "skip_batch_stride": ("const double a = Ad[b * strideA", "const double a = Ad[0 * strideA"),
    "not_zeroed": ("r[j] = 0.0;", "r[j] = r[j] * 1.0 + 1.0;"),
    "q4_nibble_order": ("(row[k / 8] >> (4 * (k % 8)))", "(row[k / 8] >> (4 * (7 - k % 8)))"),
    "q4_zero_point": ("((double)q - 8.0)", "((double)q - 7.0)"),
    "q4_group_index": ("srow[k / G]", "srow[(k / G + 1) % ((K + G - 1) / G)]"),
    "q4_wrong_row": ("Wq + n * ldq", "Wq + ((n + 1) % N) * ldq"),
    "q4_scale_row": ("S + n * lds", "S + ((n + 1) % N) * lds"),
}


def _pin_batched(o):
    """Batched operands: each slice is its own product (exact integers)."""
    A, B = workloads.small_int_operands(5, 4, 6, 9, 7, "f32")
    exact = np.matmul(A.astype(np.int64), B.astype(np.int64)).astype(np.float64)
    assert np.array_equal(o.matmul(A, B), exact)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc needed to build mutants")
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(tmp_path, name):
    src = open(oracle._SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    path = tmp_path / f"oracle_{name}.c"
    path.write_text(src.replace(old, new))
    so = oracle.build(force=True, src=str(path), out=str(tmp_path / f"lib_{name}.so"))
    mutant = oracle.Oracle(so)
    failed = []
    for pin in PINS + [_pin_batched]:
        try:
            pin(mutant)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"no pin caught the planted mistake {name}"
