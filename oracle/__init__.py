"""CPU oracle for C = A . B -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and never imports it.

``matmul`` evaluates the plain definition of the paper's MatMul /
BatchMatMul (kernel table, Table 3; a candidate kernel is only a schedule of
this loop nest, Sec. 2 and Fig. 10): R[b,i,j] = sum_k A[b,i,k] * B[b,k,j] in
fp64, k ascending, in the C file ``oracle.c`` (built with gcc, OpenMP).
Results are fp64 numpy arrays.

Every function here is pinned by ``tests/test_oracle_pins.py`` against
identities, permutations, closed forms, exact integer and exact rational
arithmetic, and numpy's float64 product.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

F32, F16 = 0, 1


def build(force: bool = False, src: str = _SRC, out: str = _LIB) -> str:
    """Compile ``oracle.c`` (or another source, e.g. a planted-mistake copy in
    a test) into a shared library with gcc: -O2, no fast-math, no FP
    contraction."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
               "-fno-fast-math", "-std=c11", src, "-o", tmp]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.float16:
        return F16
    raise TypeError(f"oracle takes float32 or float16 operands, got {a.dtype}")


def _as3(x: np.ndarray) -> np.ndarray:
    return x[None] if x.ndim == 2 else x


class Oracle:
    """ctypes binding of one build of ``oracle.c``."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        i64, vp = ctypes.c_int64, ctypes.c_void_p
        lib.oracle_matmul.restype = ctypes.c_int
        lib.oracle_matmul.argtypes = [i64, i64, i64, i64, vp, i64, i64, vp, i64, i64,
                                      vp, i64, i64, ctypes.c_int, ctypes.c_int]
        lib.oracle_f16_to_f64.restype = ctypes.c_double
        lib.oracle_f16_to_f64.argtypes = [ctypes.c_uint16]
        lib.oracle_max_threads.restype = ctypes.c_int
        lib.oracle_gemv_q4.restype = ctypes.c_int
        lib.oracle_gemv_q4.argtypes = [i64, i64, vp, vp, i64, vp, i64, i64, vp, ctypes.c_int]
        self.lib = lib

    def matmul(self, A: np.ndarray, B: np.ndarray, nthreads: int = 0) -> np.ndarray:
        """fp64 product of row-major A[(b,)M,K] and B[(b,)K,N] (same dtype)."""
        if A.dtype != B.dtype:
            raise TypeError("A and B must share a dtype")
        squeeze = A.ndim == 2 and B.ndim == 2
        A3 = np.ascontiguousarray(_as3(A))
        B3 = np.ascontiguousarray(_as3(B))
        batch, M, K = A3.shape
        if B3.shape[0] != batch or B3.shape[1] != K:
            raise ValueError(f"shape mismatch {A.shape} . {B.shape}")
        N = B3.shape[2]
        R = np.empty((batch, M, N), dtype=np.float64)
        rc = self.lib.oracle_matmul(batch, M, N, K, A3.ctypes.data, K, M * K,
                                    B3.ctypes.data, N, K * N, R.ctypes.data, N, M * N,
                                    _dtype_code(A3), int(nthreads))
        if rc != 0:
            raise RuntimeError(f"oracle_matmul returned {rc}")
        return R[0] if squeeze else R

    def f16_to_f64(self, bits) -> np.ndarray:
        """Decode binary16 bit patterns (uint16) to fp64, one by one."""
        bits = np.asarray(bits, dtype=np.uint16).ravel()
        return np.array([self.lib.oracle_f16_to_f64(int(b)) for b in bits], dtype=np.float64)

    def gemv_q4(self, x: np.ndarray, Wq: np.ndarray, S: np.ndarray, group: int, N: int,
                nthreads: int = 0) -> np.ndarray:
        """fp64 y[N] = x[K] . W for the 4-bit weight format of oracle.c:
        x float16 [K], Wq uint32 [N, ldq] (eight codes per word along K),
        S float16 [N, lds] (one scale per output and group of ``group``
        inputs)."""
        x = np.ascontiguousarray(x, dtype=np.float16)
        Wq = np.ascontiguousarray(Wq, dtype=np.uint32)
        S = np.ascontiguousarray(S, dtype=np.float16)
        K = x.shape[0]
        if Wq.ndim != 2 or S.ndim != 2 or Wq.shape[0] < N or S.shape[0] < N:
            raise ValueError("shape mismatch")
        if Wq.shape[1] < (K + 7) // 8 or S.shape[1] < (K + group - 1) // group:
            raise ValueError("rows too short for K")
        y = np.empty(N, dtype=np.float64)
        rc = self.lib.oracle_gemv_q4(K, N, x.ctypes.data, Wq.ctypes.data, Wq.shape[1], S.ctypes.data,
                                     S.shape[1], int(group), y.ctypes.data, int(nthreads))
        if rc != 0:
            raise RuntimeError(f"oracle_gemv_q4 returned {rc}")
        return y

    def max_threads(self) -> int:
        return int(self.lib.oracle_max_threads())


def default() -> Oracle:
    global _lib
    with _lock:
        if _lib is None:
            _lib = Oracle(build())
    return _lib


def matmul(A: np.ndarray, B: np.ndarray, nthreads: int = 0) -> np.ndarray:
    return default().matmul(A, B, nthreads)


def f16_to_f64(bits) -> np.ndarray:
    return default().f16_to_f64(bits)


def gemv_q4(x, Wq, S, group: int, N: int, nthreads: int = 0) -> np.ndarray:
    return default().gemv_q4(x, Wq, S, group, N, nthreads)


def max_threads() -> int:
    return default().max_threads()
