"""Build libnnjit.so (HIP kernels + C-ABI) for gfx950 with hipcc.

Each source is compiled to an object in parallel, then linked in-tree as
``paper_2309_08978_amd/libnnjit.so``.  All HIP code is compiled with packed
fp32 arithmetic disabled (``-packed-fp32-ops``): the kernels never rely on
v_pk_* fp32 instructions.

    python -m paper_2309_08978_amd.build          # build
    python -m paper_2309_08978_amd.build --check  # also print register use
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libnnjit.so")
OBJDIR = os.path.join(HERE, "_build")
ARCH = os.environ.get("NNJIT_ARCH", "gfx950")

SOURCES = ["gemm_f32.hip", "gemm_f16.hip", "gemv.hip", "gemv_q4.hip", "noalloc.hip", "space.cpp", "runtime.cpp"]

COMMON = ["-O3", "-fPIC", "-std=c++17", "-Wall", "-Wno-unused-function",
          "-I", CSRC, "-I", os.path.join(ROOT, "include")]
DEVICE = ["-x", "hip", f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(src: str, resource_usage: bool) -> tuple[str, str, float]:
    t0 = time.time()
    obj = os.path.join(OBJDIR, src + ".o")
    cmd = [hipcc()] + COMMON
    if src.endswith(".hip"):
        cmd += DEVICE
        if resource_usage:
            cmd += ["-Rpass-analysis=kernel-resource-usage"]
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"compile of {src} failed:\n{' '.join(cmd)}\n{p.stdout}\n{p.stderr}")
    return obj, p.stderr, time.time() - t0


def build(verbose: bool = False, resource_usage: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    jobs = min(len(SOURCES), int(os.environ.get("MAX_JOBS", "8")), 16)
    objs, logs = [], {}
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = {ex.submit(_compile, s, resource_usage): s for s in SOURCES}
        for f in cf.as_completed(futs):
            obj, err, dt = f.result()
            logs[futs[f]] = err
            if verbose:
                print(f"  {futs[f]}: {dt:.1f}s", flush=True)
    objs = [os.path.join(OBJDIR, s + ".o") for s in SOURCES]
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{p.stdout}\n{p.stderr}")
    os.replace(tmp, LIB)
    if resource_usage:
        for s in SOURCES:
            if logs.get(s):
                print(logs[s])
    return LIB


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--check", action="store_true", help="print per-kernel resource usage")
    a = ap.parse_args(argv)
    t0 = time.time()
    lib = build(verbose=True, resource_usage=a.check)
    print(f"built {lib} in {time.time() - t0:.1f}s")
    return 0


if __name__ == "__main__":
    sys.exit(main())
