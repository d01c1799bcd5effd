"""Builds libcelty.so in-tree with hipcc for gfx950.

Usage: python paper_2608_01536_amd/build_lib.py   (or __graft_entry__.build()).
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libcelty.so")
SOURCES = [os.path.join(PKG, "csrc", "spmspv.hip"), os.path.join(PKG, "csrc", "select.hip"),
           os.path.join(PKG, "csrc", "encode.cpp"),
           # a measurement reference for the benchmark (include/celty_bench.h)
           os.path.join(PKG, "csrc", "bench_read.hip")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
    # packed fp32 VALU forms stay off (the compiler must not emit v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # the leading kernel arguments (those a workgroup's prologue needs: the
    # selection's pointers and sizes, the column maxima, R and M; nine
    # arguments in 12 scalar registers) are preloaded at dispatch instead of
    # fetched from memory
    "-Xarch_device", "-mllvm=-amdgpu-kernarg-preload-count=13",
    "-I", os.path.join(ROOT, "include"), "-pthread",
]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, "-o", tmp, *SOURCES]
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
