"""Build step: generate the per-variant device code, then compile libe3mi.so.

1. g++ builds the table generator (csrc/gen.cpp + csrc/builder.cpp) and runs
   it, writing csrc/generated/variants.inc (coupling constants as literals).
2. hipcc compiles the HIP kernels, the C ABI and the builder into
   libe3mi.so for gfx950, next to this file.

Run: python -m paper_2609_35099_amd.build  (or __graft_entry__.build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libe3mi.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed-FP32 instructions are disabled for every HIP translation unit.
HIP_FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-fPIC", "-Wno-unused-command-line-argument"]


def _run(cmd, verbose):
    if verbose:
        print("+", " ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"build step failed: {cmd[0]} (exit {res.returncode})")
    return res


def build(verbose: bool = True) -> str:
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(os.path.join(CSRC, "generated"), exist_ok=True)
    gen = os.path.join(BUILD, "e3gen")
    _run(["g++", "-O2", "-std=c++17", "-o", gen,
          os.path.join(CSRC, "gen.cpp"), os.path.join(CSRC, "builder.cpp")], verbose)
    inc = os.path.join(CSRC, "generated", "variants.inc")
    tmp = inc + ".tmp"
    _run([gen, tmp], verbose)
    if not os.path.exists(inc) or open(inc).read() != open(tmp).read():
        shutil.move(tmp, inc)
    else:
        os.remove(tmp)
    out_tmp = LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-shared", "-o", out_tmp,
          os.path.join(CSRC, "e3mi.hip"), os.path.join(CSRC, "builder.cpp")], verbose)
    os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
