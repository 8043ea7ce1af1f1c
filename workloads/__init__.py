"""Seeded synthetic inputs for the dense MatMul / BatchMatMul / GEMV workloads.

This module only draws numbers and describes shapes. It holds none of the
method's arithmetic, so both the HIP path (through its tests and bench) and
the CPU oracle may take their inputs from here.

Shapes are transformer-layer shapes: the paper evaluates MatMul and
BatchMatMul kernels picked from transformer models (Table 3: K0-K3; Sec. 7.1
"Kernels and models") and writes a MatMul shape as [M, K, N].  Every op here
keeps that order: ``Op.M, Op.K, Op.N``; C[M, N] = A[M, K] . B[K, N], all
row-major, ``batch`` independent products for a BatchMatMul.

Value recipes (the paper uses no dataset; model-shaped synthetic values stand
in for real weights and activations):

* ``u11``      i.i.d. uniform [-1, 1) in fp32
* ``act``      activations, N(0, 1)
* ``w``        weights, N(0, 0.02)
* ``softmax``  attention probabilities: each row is the softmax of N(0, 1)
               logits (computed in fp64, then rounded to the input dtype)
* ``causal``   as ``softmax`` but logits with j > i are -inf (upper triangle 0)
* ``int8``     small integers uniform in {-8..8}; every partial sum of a
               product of such matrices is an integer below 2^24, so any
               summation order gives the same fp32 result

4-bit weight-only GEMV (dtype ``q4``; the paper's Llama-2-7B decode runs on
4-bit weights, Sec. 7, without giving the format): x fp16 [K]; the weight
is stored as a linear layer's weight, one row per output: codes are 32-bit
words [N][ldq], eight 4-bit codes per word along K, drawn as uniformly
random words (every code uniform in 0..15); one fp16 scale per output and
group of ``group`` inputs ([N][lds]), uniform in [0.002, 0.01) -- the size of
max|w| / 7 over a 128-input group of N(0, 0.02) weights.  The exact-arithmetic
recipe (``q4_int``) takes x in {-8..8} and scales in {1/2, 1, 2, 4}: every
partial sum is then a multiple of 1/2 below 2^23, exact in fp32.

fp16 inputs are drawn in fp32 and rounded once, round-to-nearest-even
(numpy ``astype(float16)``); the GPU and the oracle consume the same bits.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np

F32 = "f32"
F16 = "f16"
Q4 = "q4"
_NP = {F32: np.float32, F16: np.float16}


@dataclasses.dataclass(frozen=True)
class Op:
    """One product C[batch][M, N] = A[batch][M, K] . B[batch][K, N]."""

    name: str
    M: int
    K: int
    N: int
    batch: int = 1
    a_dist: str = "act"
    b_dist: str = "w"
    dtype: str = F32
    group: int = 0          # q4: rows per scale group

    @property
    def kind(self) -> str:
        if self.dtype == Q4:
            return "gemv_q4"
        if self.batch > 1:
            return "batched"
        return "gemv" if self.M == 1 else "gemm"

    @property
    def flops(self) -> int:
        return 2 * self.batch * self.M * self.N * self.K

    @property
    def elt(self) -> int:
        return 2 if self.dtype == F16 else 4

    @property
    def weight_bytes(self) -> int:
        """Bytes of the B operand (q4: code words plus scales)."""
        if self.dtype == Q4:
            return self.N * (-(-self.K // 8)) * 4 + self.N * (-(-self.K // self.group)) * 2
        return self.batch * self.K * self.N * self.elt

    @property
    def bytes(self) -> int:
        """Compulsory HBM bytes: read A and B once, write fp32 C once."""
        if self.dtype == Q4:
            return self.K * 2 + self.weight_bytes + self.N * 4
        return self.batch * ((self.M * self.K + self.K * self.N) * self.elt + self.M * self.N * 4)

    def with_dtype(self, dtype: str) -> "Op":
        return dataclasses.replace(self, dtype=dtype)


def _linears(prefix: str, M: int, shapes: List[Tuple[str, int, int]]) -> List[Op]:
    return [Op(f"{prefix}.{n}", M, K, N) for (n, K, N) in shapes]


def _bart_base_seq128() -> List[Op]:
    # BART-base encoder layer, d_model 768, d_ff 3072, 12 heads of 64, seq 128
    ops = _linears("bart", 128, [("qkv", 768, 2304), ("out_proj", 768, 768),
                                 ("ffn_up", 768, 3072), ("ffn_down", 3072, 768)])
    ops += [Op("bart.attn_qk", 128, 64, 128, batch=12, a_dist="act", b_dist="act"),
            Op("bart.attn_pv", 128, 128, 64, batch=12, a_dist="softmax", b_dist="act")]
    return ops


def _t5_large_b4s256() -> List[Op]:
    # T5-large encoder layer, d_model 1024, d_ff 4096, 16 heads of 64, batch 4 x seq 256
    ops = _linears("t5", 1024, [("q", 1024, 1024), ("k", 1024, 1024), ("v", 1024, 1024),
                                ("o", 1024, 1024), ("ffn_up", 1024, 4096), ("ffn_down", 4096, 1024)])
    ops += [Op("t5.attn_qk", 256, 64, 256, batch=64, a_dist="act", b_dist="act"),
            Op("t5.attn_pv", 256, 256, 64, batch=64, a_dist="softmax", b_dist="act")]
    return ops


_LLAMA_LIN = [("qkv", 4096, 12288), ("o", 4096, 4096), ("gate", 4096, 11008),
              ("up", 4096, 11008), ("down", 11008, 4096), ("lm_head", 4096, 32000)]


def _llama_decode(dtype: str) -> List[Op]:
    return [dataclasses.replace(op, dtype=dtype) for op in _linears("llama.decode", 1, _LLAMA_LIN)]


def _llama_prefill(dtype: str) -> List[Op]:
    lin = [s for s in _LLAMA_LIN if s[0] != "up"]  # gate and up share a shape; listed once
    ops = _linears("llama.prefill", 512, lin)
    ops += [Op("llama.attn_qk", 512, 128, 512, batch=32, a_dist="act", b_dist="act"),
            Op("llama.attn_pv", 512, 512, 128, batch=32, a_dist="causal", b_dist="act")]
    return [dataclasses.replace(op, dtype=dtype) for op in ops]


def _llama_decode_q4(group: int) -> List[Op]:
    return [dataclasses.replace(op, dtype=Q4, group=group) for op in _linears("llama.decode", 1, _LLAMA_LIN)]


def _paper_kernels() -> List[Op]:
    # Table 3 of the paper: K0 RoBERTa, K1 GPT-2 MatMuls; K2 BART, K3 GPT-2 BatchMatMuls
    return [Op("K0", 384, 768, 768), Op("K1", 640, 768, 3072),
            Op("K2", 384, 384, 64, batch=12, a_dist="softmax", b_dist="act"),
            Op("K3", 64, 64, 64, batch=120, a_dist="act", b_dist="act")]


#: Named workloads. Index 0..4 follow the order the workloads are listed in
#: the build's configuration table; the seed of every op derives from it.
WORKLOADS: Dict[str, Tuple[int, List[Op]]] = {
    "matmul_64x768x768_f32": (0, [Op("single", 64, 768, 768, a_dist="u11", b_dist="u11")]),
    "bart_base_layer_seq128_f32": (1, _bart_base_seq128()),
    "t5_large_layer_b4s256_f32": (2, _t5_large_b4s256()),
    "llama2_7b_decode_f32": (3, _llama_decode(F32)),
    "llama2_7b_decode_f16": (3, _llama_decode(F16)),
    "llama2_7b_decode_q4": (3, _llama_decode_q4(128)),
    "llama2_7b_prefill512_f32": (4, _llama_prefill(F32)),
    "llama2_7b_prefill512_f16": (4, _llama_prefill(F16)),
    "paper_table3_f32": (5, _paper_kernels()),
}


def workload(name: str) -> List[Op]:
    return WORKLOADS[name][1]


def _rng_for(name: str, op_index: int, role: int) -> np.random.Generator:
    wl_index = WORKLOADS[name][0]
    return np.random.default_rng([wl_index, op_index, role])


def _draw(rng: np.random.Generator, dist: str, shape: Tuple[int, ...]) -> np.ndarray:
    """fp32 values of one operand, shape (..., rows, cols)."""
    if dist == "u11":
        return rng.random(shape, dtype=np.float32) * np.float32(2) - np.float32(1)
    if dist == "act":
        return rng.standard_normal(shape, dtype=np.float32)
    if dist == "w":
        return rng.standard_normal(shape, dtype=np.float32) * np.float32(0.02)
    if dist in ("softmax", "causal"):
        logits = rng.standard_normal(shape).astype(np.float64)
        if dist == "causal":
            r, c = shape[-2], shape[-1]
            mask = np.triu(np.ones((r, c), dtype=bool), k=1)
            logits = np.where(mask, -np.inf, logits)
        logits = logits - logits.max(axis=-1, keepdims=True)
        e = np.exp(logits)
        return (e / e.sum(axis=-1, keepdims=True)).astype(np.float32)
    if dist == "int8":
        return rng.integers(-8, 9, size=shape).astype(np.float32)
    raise ValueError(f"unknown distribution {dist!r}")


def _shape(batch: int, rows: int, cols: int) -> Tuple[int, ...]:
    return (batch, rows, cols) if batch > 1 else (rows, cols)


def op_inputs(name: str, op_index: int) -> Tuple[np.ndarray, ...]:
    """(A, B) for op ``op_index`` of workload ``name``: contiguous row-major
    arrays in the op's dtype. A is [batch,]M x K, B is [batch,]K x N.
    A q4 op gives (x, Wq, scales) as ``q4_operands`` does."""
    op = workload(name)[op_index]
    if op.dtype == Q4:
        return q4_operands(_rng_for(name, op_index, 0), op.K, op.N, op.group)
    if WORKLOADS[name][0] == 0:
        # the single 64x768x768 product: one generator seeded 0, A drawn first, then B
        rng = np.random.default_rng(0)
        a = _draw(rng, op.a_dist, _shape(op.batch, op.M, op.K))
        b = _draw(rng, op.b_dist, _shape(op.batch, op.K, op.N))
    else:
        a = _draw(_rng_for(name, op_index, 0), op.a_dist, _shape(op.batch, op.M, op.K))
        b = _draw(_rng_for(name, op_index, 1), op.b_dist, _shape(op.batch, op.K, op.N))
    t = _NP[op.dtype]
    return np.ascontiguousarray(a.astype(t)), np.ascontiguousarray(b.astype(t))


def random_operands(seed, batch: int, M: int, K: int, N: int, dtype: str = F32,
                    a_dist: str = "act", b_dist: str = "w") -> Tuple[np.ndarray, np.ndarray]:
    """Operands for an arbitrary (test) shape from ``default_rng(seed)``;
    A is drawn first, then B. Arrays are 3-D when ``batch`` > 1."""
    rng = np.random.default_rng(seed)
    a = _draw(rng, a_dist, _shape(batch, M, K))
    b = _draw(rng, b_dist, _shape(batch, K, N))
    t = _NP[dtype]
    return np.ascontiguousarray(a.astype(t)), np.ascontiguousarray(b.astype(t))


def small_int_operands(seed, batch: int, M: int, K: int, N: int,
                       dtype: str = F32) -> Tuple[np.ndarray, np.ndarray]:
    """Entries uniform in {-8..8}: all partial sums are exact in fp32."""
    return random_operands(seed, batch, M, K, N, dtype, a_dist="int8", b_dist="int8")


def q4_operands(seed, K: int, N: int, group: int, ldq: int | None = None, lds: int | None = None,
                recipe: str = "q4") -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """(x fp16 [K], Wq uint32 [N, ldq], scales fp16 [N, lds]) for a 4-bit
    weight-only GEMV, from ``default_rng(seed)`` (or a Generator): x first,
    then the code words, then the scales.  ``ldq`` defaults to ceil(K / 8) and
    ``lds`` to ceil(K / group); padding words and scales are random too.
    recipe ``q4``: x N(0, 1), scales uniform [0.002, 0.01); ``q4_int``: x in
    {-8..8}, scales in {1/2, 1, 2, 4} (every partial sum is exact in fp32
    for K below 2^16)."""
    rng = seed if isinstance(seed, np.random.Generator) else np.random.default_rng(seed)
    ldq = -(-K // 8) if ldq is None else ldq
    ngroups = -(-K // group)
    lds = ngroups if lds is None else lds
    if recipe == "q4":
        x = rng.standard_normal(K, dtype=np.float32).astype(np.float16)
    elif recipe == "q4_int":
        x = rng.integers(-8, 9, size=K).astype(np.float16)
    else:
        raise ValueError(f"unknown q4 recipe {recipe!r}")
    Wq = rng.integers(0, 1 << 32, size=(N, ldq), dtype=np.uint32)
    if recipe == "q4":
        S = (rng.random((N, lds), dtype=np.float32) * np.float32(0.008) + np.float32(0.002)).astype(np.float16)
    else:
        S = rng.choice(np.array([0.5, 1.0, 2.0, 4.0], dtype=np.float16), size=(N, lds))
    return np.ascontiguousarray(x), np.ascontiguousarray(Wq), np.ascontiguousarray(S)
