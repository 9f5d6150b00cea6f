"""Build libentropack.so in-tree for gfx950.

Host sources (encoder, blob validation) are compiled with g++, the kernels
with hipcc for gfx950 only; hipcc links the shared library.  Packed FP32 VALU
forms are disabled for all device code; floating-point contraction is off so
the encoder's arithmetic is the plain IEEE sequence written in the source.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(os.path.dirname(HERE), "_build")
LIB = os.path.join(HERE, "libentropack.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

HOST_SRC = ["encode.cpp", "capi.cpp"]
HIP_SRC = ["decode.hip", "decode_args.hip", "decode_mixed.hip", "decode_gemm.hip", "gemm_i8.hip", "encode_gpu.hip"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off"]
HIP_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-munsafe-fp-atomics"]


def _run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)


def build(verbose: bool = True) -> str:
    """Compile every source (concurrently: each decode source takes minutes) and link."""
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    for src in HOST_SRC:
        obj = os.path.join(BUILD, src + ".o")
        jobs.append((["g++", *COMMON, "-pthread", "-Wall", "-c", os.path.join(CSRC, src), "-o", obj], obj))
    for src in HIP_SRC:
        path = os.path.join(CSRC, src)
        if not os.path.exists(path):
            continue
        obj = os.path.join(BUILD, src + ".o")
        jobs.append(([HIPCC, *COMMON, *HIP_FLAGS, "-c", path, "-o", obj], obj))
    with ThreadPoolExecutor(max_workers=len(jobs)) as pool:
        for f in [pool.submit(_run, cmd) for cmd, _ in jobs]:
            f.result()
    objs = [obj for _, obj in jobs]
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-pthread", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
