"""Acceptance check of a GPU result against the oracle -- TEST INFRASTRUCTURE.

The bar is the one the product is held to:

* fp32 inputs: relative Frobenius error ||C - R||_F / ||R||_F <= 1e-5 AND every
  element |C - R| <= 2e-6 * K * max|A| * max|B| (maxima over the whole A and B).
* fp16 inputs (fp32 accumulate): relative Frobenius error <= 2e-3.
* ||R||_F == 0 (or a zero per-element bound) requires C == 0 exactly.
* any NaN or Inf in C fails; comparisons are written ``not (err <= bound)``.

Everything is evaluated in fp64 on the host over all elements (all batches).
"""
from __future__ import annotations

import numpy as np

REL_FRO = {"f32": 1e-5, "f16": 2e-3}
ELT_COEF = 2e-6


def check(C, R, A, B, dtype: str, K: int | None = None) -> dict:
    C = np.asarray(C, dtype=np.float64)
    R = np.asarray(R, dtype=np.float64)
    if C.shape != R.shape:
        raise ValueError(f"shape mismatch {C.shape} vs {R.shape}")
    A64 = np.asarray(A, dtype=np.float64)
    B64 = np.asarray(B, dtype=np.float64)
    if K is None:
        K = A64.shape[-1]
    finite = bool(np.all(np.isfinite(C)))
    diff = C - R
    nr = float(np.sqrt(np.sum(R * R)))
    nd = float(np.sqrt(np.sum(diff * diff))) if finite else float("inf")
    amax = float(np.max(np.abs(A64))) if A64.size else 0.0
    bmax = float(np.max(np.abs(B64))) if B64.size else 0.0
    elt_bound = ELT_COEF * K * amax * bmax
    max_err = float(np.max(np.abs(diff))) if diff.size and finite else (0.0 if finite else float("inf"))
    if nr == 0.0:
        rel = 0.0 if (finite and not np.any(C != 0)) else float("inf")
    else:
        rel = nd / nr
    ok = finite and (rel <= REL_FRO[dtype])
    if dtype == "f32":
        if elt_bound == 0.0:
            ok = ok and not np.any(C != 0)
        else:
            ok = ok and (max_err <= elt_bound)
    return {"ok": bool(ok), "rel_fro": rel, "max_err": max_err, "elt_bound": elt_bound,
            "finite": finite, "K": K}

