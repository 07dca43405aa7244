"""Build libstmoe.so (HIP kernels + C ABI) for gfx950 in-tree.

    python -m paper_2606_15453_amd.build        # or build() from Python

Every HIP translation unit is compiled with packed-fp32 instructions
disabled; objects go to ``_build/`` next to this file and the library to
``libstmoe.so`` beside it.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = ["util.cpp", "route_topk.hip", "predictor.hip", "expert_ffn.hip", "expert_cache.cpp",
           "cache_device.hip", "decode_layer.hip", "calib.hip"]
LIB = os.path.join(HERE, "libstmoe.so")
ARCH = "gfx950"


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def _flags():
    return ["-O3", "-fPIC", "-std=c++17", f"--offload-arch={ARCH}", "-mcode-object-version=5",
            "-Wall", "-Wno-unused-result",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include")]


def _compile(src: str, obj: str) -> str:
    cmd = [_hipcc()] + _flags() + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    out = os.path.join(HERE, "_build")
    os.makedirs(out, exist_ok=True)
    jobs = []
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        for s in SOURCES:
            src = os.path.join(HERE, "csrc", s)
            obj = os.path.join(out, os.path.splitext(s)[0] + ".o")
            jobs.append(ex.submit(_compile, src, obj))
        objs = [j.result() for j in jobs]
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
