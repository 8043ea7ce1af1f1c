"""Python binding of libnnjit (include/nnjit.h): argument marshalling only.

Every ``nnjit_*`` function here has the name and argument order of the C
entry point it calls and returns its integer code unchanged; pointer
arguments accept a ``torch.Tensor`` (its ``data_ptr()``), an int or None, and
``stream`` accepts a ``torch.cuda.Stream``, an int handle or None.  All the
work runs in the HIP library; if ``libnnjit.so`` is missing the binding
raises instead of falling back to anything else.

``matmul`` / ``batched_matmul`` are conveniences that take tensors, derive
(M, N, K), leading dimensions and batch strides from them, call the entry
point and raise ``NnjitError`` on a negative code.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnnjit.so")

NNJIT_F32, NNJIT_F16 = 0, 1
NNJIT_KIND_GEMM, NNJIT_KIND_BATCHED, NNJIT_KIND_GEMV, NNJIT_KIND_GEMV_Q4 = 0, 1, 2, 3
NNJIT_OK, NNJIT_EINVAL, NNJIT_EDTYPE, NNJIT_ENOCFG, NNJIT_EHIP, NNJIT_ENOMEM = 0, -1, -2, -3, -4, -5
ERROR_NAMES = {-1: "NNJIT_EINVAL", -2: "NNJIT_EDTYPE", -3: "NNJIT_ENOCFG", -4: "NNJIT_EHIP", -5: "NNJIT_ENOMEM"}

EXPORTED = ["nnjit_matmul", "nnjit_batched_matmul", "nnjit_batched_matmul_noalloc", "nnjit_tune", "nnjit_tune_batched", "nnjit_matmul_config",
            "nnjit_gemv_q4", "nnjit_tune_gemv_q4", "nnjit_gemv_q4_config",
            "nnjit_num_configs", "nnjit_config_info", "nnjit_config_resources", "nnjit_lite_space",
            "nnjit_last_tune_stats", "nnjit_last_tune_stats_ex", "nnjit_last_tune_trace", "nnjit_cached_config", "nnjit_cached_ranked",
            "nnjit_set_online", "nnjit_online_status", "nnjit_cache_clear",
            "nnjit_cache_save", "nnjit_cache_load", "nnjit_stream_read", "nnjit_last_error", "nnjit_version"]


class NnjitError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


class DeviceLimits(ctypes.Structure):
    _fields_ = [("num_cus", ctypes.c_int), ("simds_per_cu", ctypes.c_int), ("vgprs_per_lane", ctypes.c_int),
                ("vgpr_granule", ctypes.c_int), ("max_waves_per_simd", ctypes.c_int), ("wave_size", ctypes.c_int),
                ("lds_per_cu", ctypes.c_int64), ("lds_per_wg", ctypes.c_int64), ("max_threads_per_wg", ctypes.c_int)]


class Resources(ctypes.Structure):
    _fields_ = [("regs_per_lane", ctypes.c_int), ("regs_measured", ctypes.c_int), ("lds_per_wg", ctypes.c_int64),
                ("threads_per_wg", ctypes.c_int), ("waves_per_wg", ctypes.c_int), ("reg_limit", ctypes.c_int),
                ("lds_limit", ctypes.c_int), ("wave_limit", ctypes.c_int), ("wg_per_cu", ctypes.c_int)]


class TuneStats(ctypes.Structure):
    _fields_ = [("wall_ms", ctypes.c_double), ("eval_ms", ctypes.c_double), ("n_enumerated", ctypes.c_int),
                ("n_lite", ctypes.c_int), ("n_timed", ctypes.c_int), ("n_aborted", ctypes.c_int),
                ("n_failed", ctypes.c_int), ("chosen", ctypes.c_int), ("best_us", ctypes.c_double),
                ("default_us", ctypes.c_double), ("cache_hit", ctypes.c_int)]


def mi355x_limits() -> DeviceLimits:
    """MI355X constants for the host-only resource model."""
    return DeviceLimits(256, 4, 512, 8, 8, 64, 163840, 163840, 1024)


_lock = threading.Lock()
_lib = None


def load(build_if_missing: bool = False) -> ctypes.CDLL:
    """Load libnnjit.so (built in-tree by ``paper_2309_08978_amd.build``)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            if not build_if_missing:
                raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2309_08978_amd.build`")
            from . import build as _b
            _b.build()
        lib = ctypes.CDLL(LIB_PATH)
        i64, vp, ci = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        sig = {
            "nnjit_matmul": [i64, i64, i64, vp, i64, vp, i64, vp, i64, ci, vp],
            "nnjit_batched_matmul": [i64, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64, ci, vp],
            "nnjit_batched_matmul_noalloc": [i64, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64, ci, vp],
            "nnjit_tune": [i64, i64, i64, ci],
            "nnjit_tune_batched": [i64, i64, i64, i64, ci],
            "nnjit_matmul_config": [ci, i64, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64, ci, vp],
            "nnjit_gemv_q4": [i64, i64, i64, vp, vp, i64, vp, i64, vp, vp],
            "nnjit_tune_gemv_q4": [i64, i64, i64],
            "nnjit_gemv_q4_config": [ci, i64, i64, i64, vp, vp, i64, vp, i64, vp, vp],
            "nnjit_num_configs": [],
            "nnjit_config_info": [ci, ctypes.c_char_p, i64],
            "nnjit_config_resources": [ci, ctypes.POINTER(DeviceLimits), ctypes.POINTER(Resources)],
            "nnjit_lite_space": [ci, ci, i64, i64, i64, i64, ctypes.POINTER(DeviceLimits),
                                 ctypes.POINTER(ci), ci, ctypes.POINTER(ci), ctypes.POINTER(i64)],
            "nnjit_last_tune_stats": [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ci), ctypes.POINTER(ci),
                                      ctypes.POINTER(ci)],
            "nnjit_last_tune_stats_ex": [ctypes.POINTER(TuneStats)],
            "nnjit_last_tune_trace": [ctypes.POINTER(ci), ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(ctypes.c_double), ci],
            "nnjit_cached_config": [ci, ci, i64, i64, i64, i64],
            "nnjit_cached_ranked": [ci, ci, i64, i64, i64, i64, ctypes.POINTER(ci), ctypes.POINTER(ctypes.c_double), ci],
            "nnjit_set_online": [ci],
            "nnjit_online_status": [ci, ci, i64, i64, i64, i64, ctypes.POINTER(ci), ctypes.POINTER(ci),
                                    ctypes.POINTER(ci)],
            "nnjit_cache_clear": [],
            "nnjit_cache_save": [ctypes.c_char_p],
            "nnjit_cache_load": [ctypes.c_char_p],
            "nnjit_stream_read": [vp, i64, vp, ci, vp],
            "nnjit_last_error": [],
            "nnjit_version": [],
        }
        for name, args in sig.items():
            f = getattr(lib, name)
            f.argtypes = args
            f.restype = ctypes.c_char_p if name == "nnjit_last_error" else ctypes.c_int
        _lib = lib
        return lib


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


# ------------------------------------------------------ entry points (1:1)

def nnjit_matmul(M, N, K, A, lda, B, ldb, C, ldc, dtype, stream=None) -> int:
    return load().nnjit_matmul(M, N, K, _ptr(A), lda, _ptr(B), ldb, _ptr(C), ldc, dtype, _stream(stream))


def nnjit_batched_matmul(batch, M, N, K, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, dtype,
                         stream=None) -> int:
    return load().nnjit_batched_matmul(batch, M, N, K, _ptr(A), lda, strideA, _ptr(B), ldb, strideB,
                                       _ptr(C), ldc, strideC, dtype, _stream(stream))


def nnjit_batched_matmul_noalloc(batch, M, N, K, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, dtype,
                                 stream=None) -> int:
    return load().nnjit_batched_matmul_noalloc(batch, M, N, K, _ptr(A), lda, strideA, _ptr(B), ldb, strideB,
                                               _ptr(C), ldc, strideC, dtype, _stream(stream))


def nnjit_tune(M, N, K, dtype) -> int:
    return load().nnjit_tune(M, N, K, dtype)


def nnjit_tune_batched(batch, M, N, K, dtype) -> int:
    return load().nnjit_tune_batched(batch, M, N, K, dtype)


def nnjit_matmul_config(cfg, batch, M, N, K, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, dtype,
                        stream=None) -> int:
    return load().nnjit_matmul_config(cfg, batch, M, N, K, _ptr(A), lda, strideA, _ptr(B), ldb, strideB,
                                      _ptr(C), ldc, strideC, dtype, _stream(stream))


def nnjit_gemv_q4(N, K, group, x, Wq, ldq, scales, lds, y, stream=None) -> int:
    return load().nnjit_gemv_q4(N, K, group, _ptr(x), _ptr(Wq), ldq, _ptr(scales), lds, _ptr(y), _stream(stream))


def nnjit_tune_gemv_q4(N, K, group) -> int:
    return load().nnjit_tune_gemv_q4(N, K, group)


def nnjit_gemv_q4_config(cfg, N, K, group, x, Wq, ldq, scales, lds, y, stream=None) -> int:
    return load().nnjit_gemv_q4_config(cfg, N, K, group, _ptr(x), _ptr(Wq), ldq, _ptr(scales), lds, _ptr(y),
                                       _stream(stream))


def nnjit_num_configs() -> int:
    return load().nnjit_num_configs()


def nnjit_config_info(cfg) -> str:
    buf = ctypes.create_string_buffer(512)
    rc = load().nnjit_config_info(cfg, buf, len(buf))
    if rc < 0:
        raise NnjitError(rc, nnjit_last_error())
    return buf.value.decode()


def nnjit_config_resources(cfg, dev: Optional[DeviceLimits] = None) -> dict:
    out = Resources()
    rc = load().nnjit_config_resources(cfg, ctypes.byref(dev) if dev is not None else None, ctypes.byref(out))
    if rc < 0:
        raise NnjitError(rc, nnjit_last_error())
    return {f: getattr(out, f) for f, _ in Resources._fields_}


def nnjit_lite_space(kind, dtype, batch, M, N, K, dev: Optional[DeviceLimits] = None, cap: int = 4096):
    """-> (ids in evaluation order, n_surviving, n_enumerated, n_naive)."""
    ids = (ctypes.c_int * cap)()
    n_enum = ctypes.c_int(0)
    n_naive = ctypes.c_int64(0)
    rc = load().nnjit_lite_space(kind, dtype, batch, M, N, K, ctypes.byref(dev) if dev is not None else None,
                                 ids, cap, ctypes.byref(n_enum), ctypes.byref(n_naive))
    if rc < 0:
        raise NnjitError(rc, nnjit_last_error())
    return list(ids[:min(rc, cap)]), rc, n_enum.value, n_naive.value


def nnjit_last_tune_stats() -> dict:
    """-> {'wall_ms', 'n_enum', 'n_pruned', 'n_timed'} of the last tune on this thread."""
    w = ctypes.c_double(0.0)
    e, p, t = ctypes.c_int(0), ctypes.c_int(0), ctypes.c_int(0)
    check(load().nnjit_last_tune_stats(ctypes.byref(w), ctypes.byref(e), ctypes.byref(p), ctypes.byref(t)))
    return {"wall_ms": w.value, "n_enum": e.value, "n_pruned": p.value, "n_timed": t.value}


def nnjit_last_tune_stats_ex() -> dict:
    """-> every field of nnjit_tune_stats for the last tune on this thread."""
    st = TuneStats()
    check(load().nnjit_last_tune_stats_ex(ctypes.byref(st)))
    return {f: getattr(st, f) for f, _ in TuneStats._fields_}


def nnjit_last_tune_trace(cap: int = 256):
    ids = (ctypes.c_int * cap)()
    us = (ctypes.c_double * cap)()
    at = (ctypes.c_double * cap)()
    n = load().nnjit_last_tune_trace(ids, us, at, cap)
    return [(ids[i], us[i], at[i]) for i in range(min(n, cap))]


def nnjit_cached_config(kind, dtype, batch, M, N, K) -> int:
    return load().nnjit_cached_config(kind, dtype, batch, M, N, K)


def nnjit_cached_ranked(kind, dtype, batch, M, N, K, cap: int = 5):
    """-> [(config id, us)] ranked candidates of a tuned shape (raises if not tuned)."""
    ids = (ctypes.c_int * cap)()
    us = (ctypes.c_double * cap)()
    rc = load().nnjit_cached_ranked(kind, dtype, batch, M, N, K, ids, us, cap)
    if rc < 0:
        raise NnjitError(rc, nnjit_last_error())
    return [(ids[i], us[i]) for i in range(min(rc, cap))]


def nnjit_set_online(enable: bool) -> int:
    """Switch online just-in-time tuning on or off; returns the previous setting."""
    return load().nnjit_set_online(1 if enable else 0)


def nnjit_online_status(kind, dtype, batch, M, N, K) -> dict:
    """{'state': 'online'|'tuned', 'measured', 'total', 'registered'} (raises if neither)."""
    m, t, r = ctypes.c_int(-1), ctypes.c_int(-1), ctypes.c_int(-1)
    rc = load().nnjit_online_status(kind, dtype, batch, M, N, K, ctypes.byref(m), ctypes.byref(t), ctypes.byref(r))
    if rc < 0:
        raise NnjitError(rc, nnjit_last_error())
    return {"state": "online" if rc == 0 else "tuned", "measured": m.value, "total": t.value,
            "registered": r.value}


def nnjit_cache_clear() -> int:
    return load().nnjit_cache_clear()


def nnjit_cache_save(path) -> int:
    return load().nnjit_cache_save(os.fsencode(path))


def nnjit_cache_load(path) -> int:
    return load().nnjit_cache_load(os.fsencode(path))


def nnjit_stream_read(src, nbytes, sink, workgroups, stream=None) -> int:
    return load().nnjit_stream_read(_ptr(src), nbytes, _ptr(sink), workgroups, _stream(stream))


def nnjit_last_error() -> str:
    r = load().nnjit_last_error()
    return r.decode() if r else ""


def nnjit_version() -> int:
    return load().nnjit_version()


# ------------------------------------------------------------ conveniences

def kernel_digest() -> str:
    """Short digest of the kernel and launch sources (csrc/): counter
    measurements recorded against one digest are stale under another."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(HERE, "csrc")
    for name in sorted(os.listdir(d)):
        with open(os.path.join(d, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return NNJIT_F32
    if t.dtype == torch.float16:
        return NNJIT_F16
    raise TypeError(f"unsupported dtype {t.dtype}")


def check(rc: int) -> int:
    if rc < 0:
        raise NnjitError(rc, nnjit_last_error())
    return rc


def _ld(t) -> int:
    """Leading dimension of the row-major matrices of t (last two dims):
    unit column stride, and a row stride that separates the rows."""
    rows, cols = int(t.shape[-2]), int(t.shape[-1])
    if t.stride(-1) != 1 and cols > 1:
        raise ValueError("operands must have unit stride along the last dimension")
    if rows > 1 and int(t.stride(-2)) < cols:
        raise ValueError(f"row stride {t.stride(-2)} < {cols} columns: rows overlap (an expanded or "
                         "transposed view); pass a contiguous copy")
    return max(int(t.stride(-2)), cols, 1)


def _check_operands(A, B, C, batched: bool):
    """Reject, before any library call, operands the C entry points would
    read or write out of bounds: mismatched dtypes or shapes, an output that
    is not fp32, overlapping rows or output slices, tensors not on one GPU."""
    import torch
    nd = 3 if batched else 2
    for name, t in (("A", A), ("B", B), ("C", C)):
        if t.dim() != nd:
            raise ValueError(f"{name} must be {nd}-D, got shape {tuple(t.shape)}")
    if A.dtype not in (torch.float32, torch.float16):
        raise TypeError(f"unsupported dtype {A.dtype}")
    if B.dtype != A.dtype:
        raise TypeError(f"A is {A.dtype} but B is {B.dtype}")
    if C.dtype != torch.float32:
        raise TypeError(f"C must be float32, got {C.dtype}")
    M, K = A.shape[-2:]
    K2, N = B.shape[-2:]
    if K2 != K:
        raise ValueError(f"inner dimensions differ: {tuple(A.shape)} . {tuple(B.shape)}")
    want = ((A.shape[0],) if batched else ()) + (M, N)
    if batched and B.shape[0] != A.shape[0]:
        raise ValueError(f"batch sizes differ: {tuple(A.shape)} . {tuple(B.shape)}")
    if tuple(C.shape) != want:
        raise ValueError(f"C has shape {tuple(C.shape)}, expected {want}")
    lds = [_ld(t) for t in (A, B, C)]
    if batched:
        for name, t in (("A", A), ("B", B), ("C", C)):
            if t.stride(0) < 0:
                raise ValueError(f"negative batch stride of {name}")
        span = (M - 1) * lds[2] + N if M > 0 and N > 0 else 0
        if C.shape[0] > 1 and span > 0 and C.stride(0) < span:
            raise ValueError(f"batch stride {C.stride(0)} of C < {span}: output slices overlap")
    devs = {t.device for t in (A, B, C)}
    if len(devs) != 1 or next(iter(devs)).type != "cuda":
        raise ValueError(f"A, B and C must be on one GPU, got {sorted(str(d) for d in devs)}")
    return lds


def matmul(A, B, C=None, stream=None, cfg: Optional[int] = None):
    """C = A . B for 2-D fp32/fp16 CUDA tensors (C fp32, allocated if None)."""
    import torch
    if A.dim() != 2 or B.dim() != 2:
        raise ValueError(f"matmul takes 2-D operands, got {tuple(A.shape)} . {tuple(B.shape)}")
    M, K = A.shape
    N = B.shape[1]
    if C is None:
        C = torch.empty((M, N), dtype=torch.float32, device=A.device)
    lda, ldb, ldc = _check_operands(A, B, C, batched=False)
    dt = dtype_code(A)
    if cfg is None:
        check(nnjit_matmul(M, N, K, A, lda, B, ldb, C, ldc, dt, stream))
    else:
        check(nnjit_matmul_config(cfg, 1, M, N, K, A, lda, 0, B, ldb, 0, C, ldc, 0, dt, stream))
    return C


def batched_matmul(A, B, C=None, stream=None, cfg: Optional[int] = None):
    """C[b] = A[b] . B[b] for 3-D fp32/fp16 CUDA tensors (C fp32)."""
    import torch
    if A.dim() != 3 or B.dim() != 3:
        raise ValueError(f"batched_matmul takes 3-D operands, got {tuple(A.shape)} . {tuple(B.shape)}")
    batch, M, K = A.shape
    N = B.shape[2]
    if C is None:
        C = torch.empty((batch, M, N), dtype=torch.float32, device=A.device)
    lda, ldb, ldc = _check_operands(A, B, C, batched=True)
    dt = dtype_code(A)
    sA, sB, sC = (int(t.stride(0)) for t in (A, B, C))
    if cfg is None:
        check(nnjit_batched_matmul(batch, M, N, K, A, lda, sA, B, ldb, sB, C, ldc, sC, dt, stream))
    else:
        check(nnjit_matmul_config(cfg, batch, M, N, K, A, lda, sA, B, ldb, sB, C, ldc, sC, dt, stream))
    return C


def gemv_q4(x, Wq, scales, group: int, N: int, y=None, stream=None, cfg: Optional[int] = None):
    """y = x . W for a 4-bit weight-only W (include/nnjit.h, nnjit_gemv_q4):
    x fp16 [K], Wq int32 [N, ldq] (uint32 code words, reinterpreted), scales
    fp16 [N, lds]; y fp32 [N] (allocated if None)."""
    import torch
    if x.dim() != 1 or (x.shape[0] > 1 and x.stride(0) != 1):
        raise ValueError(f"x must be a contiguous vector, got shape {tuple(x.shape)}")
    K = int(x.shape[0])
    if group < 1:
        raise ValueError(f"group must be >= 1, got {group}")
    if Wq.dim() != 2 or scales.dim() != 2 or Wq.shape[0] < N or scales.shape[0] < N:
        raise ValueError(f"shape mismatch x {tuple(x.shape)}, Wq {tuple(Wq.shape)}, scales {tuple(scales.shape)}")
    if Wq.shape[1] < -(-K // 8) or scales.shape[1] < -(-K // group):
        raise ValueError(f"rows too short for K={K}: Wq {tuple(Wq.shape)}, scales {tuple(scales.shape)}")
    if x.dtype != torch.float16 or scales.dtype != torch.float16 or Wq.element_size() != 4:
        raise TypeError("x and scales must be float16, Wq 32-bit words")
    if y is None:
        y = torch.empty((N,), dtype=torch.float32, device=x.device)
    if y.dtype != torch.float32 or tuple(y.shape) != (N,) or (N > 1 and y.stride(0) != 1):
        raise ValueError(f"y must be a contiguous float32 vector of {N}, got {y.dtype} {tuple(y.shape)}")
    devs = {t.device for t in (x, Wq, scales, y)}
    if len(devs) != 1 or next(iter(devs)).type != "cuda":
        raise ValueError(f"x, Wq, scales and y must be on one GPU, got {sorted(str(d) for d in devs)}")
    ldq, lds = _ld(Wq), _ld(scales)
    if cfg is None:
        check(nnjit_gemv_q4(N, K, group, x, Wq, ldq, scales, lds, y, stream))
    else:
        check(nnjit_gemv_q4_config(cfg, N, K, group, x, Wq, ldq, scales, lds, y, stream))
    return y


def configs() -> list:
    """Descriptions of every configuration id."""
    out = []
    for i in range(nnjit_num_configs()):
        d = {}
        for kv in nnjit_config_info(i).split():
            k, v = kv.split("=", 1)
            d[k] = int(v) if v.lstrip("-").isdigit() else v
        out.append(d)
    return out
