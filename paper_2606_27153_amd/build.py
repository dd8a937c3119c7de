"""Builds libmuon_mi355x.so (the optimizer) and libmuon_diag.so (a matrix-core
ceiling probe the bench reports as context) for gfx950 with hipcc, in-tree,
no JIT cache.

Usage: python -m paper_2606_27153_amd.build [-v]
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB_NAME = "libmuon_mi355x.so"
LIB_PATH = os.path.join(PKG, LIB_NAME)
ARCH = "gfx950"

# the GEMM kernels are instantiated in several translation units (the 256
# tile's B*X and square-output kernels per operand type, the smaller tiles)
# so that they compile in parallel
SOURCES = ["api.cpp", "plan.cpp", "ew_kernels.hip", "ns_gemm.hip", "ns_gemm_t256_bf16_bx.hip",
           "ns_gemm_t256_bf16_sq.hip", "ns_gemm_t256_f16_bx.hip", "ns_gemm_t256_f16_sq.hip", "ns_gemm_small.hip",
           "static_ws.hip"]
DIAG_SOURCES = ["diag/mfma_ceiling.hip"]
DIAG_LIB_PATH = os.path.join(PKG, "libmuon_diag.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

COMMON = [
    "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    f"--offload-arch={ARCH}",
    # no packed fp32 instructions in any device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # keep per-thread staging arrays in registers, never in LDS
    "-mllvm", "-disable-promote-alloca-to-lds",
    "-I" + os.path.join(ROOT, "include"),
    "-Wall", "-Wno-unused-result",
]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC, *COMMON, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{out}")
    if verbose and out.strip():
        print(out)
    return obj


def _link(objs, path: str, verbose: bool) -> None:
    tmp = path + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, path)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = SOURCES + DIAG_SOURCES
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 4)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    _link(objs[:len(SOURCES)], LIB_PATH, verbose)
    _link(objs[len(SOURCES):], DIAG_LIB_PATH, verbose)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
