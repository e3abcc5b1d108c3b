"""Build libglyph_tfhe.so (HIP for gfx950) in-tree with hipcc.

Usage: python -m paper_1911_07101_amd.build [-v] [--resource-usage]
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD_DIR = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libglyph_tfhe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

SOURCES = ["gt_kernels.hip", "gt_api.cpp", "gt_host.cpp", "gt_noalloc.hip", "gt_probe.hip"]
COMMON = ["-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-Wall", "-Wextra",
          "-Wno-unused-parameter", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
          # packed fp32 instructions stay off: ordinary float code only
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          # every product, sum and FMA in the kernels is written out explicitly
          "-ffp-contract=off"]


def build(verbose: bool = False, resource_usage: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs, procs = [], []
    for src in SOURCES:
        obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
        cmd = [HIPCC, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
        if resource_usage and src.endswith(".hip"):
            cmd += ["-Rpass-analysis=kernel-resource-usage"]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True))
        objs.append(obj)
    failed = False
    for src, p in zip(SOURCES, procs):
        out, _ = p.communicate()
        if out and (verbose or resource_usage or p.returncode):
            print(out, file=sys.stderr)
        if p.returncode:
            print(f"hipcc failed on {src}", file=sys.stderr)
            failed = True
    if failed:
        raise RuntimeError("HIP build failed")
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose="-v" in sys.argv, resource_usage="--resource-usage" in sys.argv)
    print(LIB)
