"""Helpers for the GPU tests: move seeded numpy operands to the device, call
the library through its C-ABI binding, bring results back as fp64."""
from __future__ import annotations

import numpy as np

import paper_2309_08978_amd as nj


def dev(x: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda:0")


def host(t) -> np.ndarray:
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().astype(np.float64)


def gpu_matmul(A: np.ndarray, B: np.ndarray, cfg=None, stream=None) -> np.ndarray:
    """C = A . B on the GPU through nnjit (tuned/default config, or a forced id)."""
    dA, dB = dev(A), dev(B)
    if A.ndim == 2:
        C = nj.matmul(dA, dB, cfg=cfg, stream=stream)
    else:
        C = nj.batched_matmul(dA, dB, cfg=cfg, stream=stream)
    return host(C)


def kind_of(batch: int, M: int) -> int:
    if batch == 1 and M == 1:
        return nj.NNJIT_KIND_GEMV
    return nj.NNJIT_KIND_GEMM if batch == 1 else nj.NNJIT_KIND_BATCHED


def dtype_code(dt: str) -> int:
    return nj.NNJIT_F16 if dt == "f16" else nj.NNJIT_F32
