"""Builds libgrpo.so (HIP, gfx950) in-tree with hipcc.

Every .hip directly under csrc/ is compiled to an object in parallel, then linked
into paper_2606_05597_amd/libgrpo.so; csrc/bench/stream_copy.hip (the
benchmark's copy ceiling) becomes libgrpo_bench.so.  Always rebuilds when called.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
SO = os.path.join(PKG, "libgrpo.so")
# the benchmark's streaming-copy ceiling, a separate library outside libgrpo's ABI
BENCH_SRC = os.path.join(CSRC, "bench", "stream_copy.hip")
BENCH_SO = os.path.join(PKG, "libgrpo_bench.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 VALU instructions are disabled on purpose: the row kernels use
# plain fp32 arithmetic throughout.
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
    "-Wall", "-Wno-unused-command-line-argument",
]


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.basename(src) + ".o")
    subprocess.check_call([HIPCC, *FLAGS, "-c", src, "-o", obj])
    return obj


def build(jobs: int = 8) -> str:
    os.makedirs(OBJ, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = SO + ".tmp"
    subprocess.check_call([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, SO)
    tmp = BENCH_SO + ".tmp"
    subprocess.check_call([HIPCC, *FLAGS, "-shared", BENCH_SRC, "-o", tmp])
    os.replace(tmp, BENCH_SO)
    return SO


if __name__ == "__main__":
    print(build())
    sys.exit(0)
