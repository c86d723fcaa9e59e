"""Build step: generate the per-variant device code, then compile libe3mi.so.

1. g++ builds the table generator (csrc/gen.cpp + csrc/builder.cpp) and runs
   it, writing csrc/generated/: variants.inc (the coupling constants of every
   compiled irreps layout as literals), one unit v_<tag>.hip per layout and
   the core unit's table of them; kinds.inc (every single x block kind of
   degree <= 3, composed at run time into other layouts), its units k_<n>.hip
   and their table.
2. hipcc compiles the core unit (csrc/e3mi.hip: C ABI, graph, linear mixing,
   record tensor product, probes), the record convolution (csrc/convr.hip:
   layouts without a compiled unit), every layout unit and the builder for
   gfx950, in parallel, and links libe3mi.so next to this file.

Layouts beyond the defaults compiled into the generator (the benchmark and
test layouts, natural-parity versions and one reordered block list) are
added with E3MI_LAYOUTS, a ';'-separated list of irreps/lmax_sh/lmax_out/parity
entries, e.g. E3MI_LAYOUTS="2e+0e+1o/3/3/all;0e+1o+1e/2/2/natural".

Run: python -m paper_2609_35099_amd.build  (or __graft_entry__.build()).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
GEN = os.path.join(CSRC, "generated")
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


def _jobs() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 4
    return max(1, min(n, int(os.environ.get("MAX_JOBS", "16")), 16))


def layouts_from_env() -> list[str]:
    return [t.strip() for t in os.environ.get("E3MI_LAYOUTS", "").split(";") if t.strip()]


def generate(verbose: bool = True, extra=None) -> list[str]:
    """Run the generator into csrc/generated; returns the layout units."""
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(GEN, exist_ok=True)
    gen = os.path.join(BUILD, "e3gen")
    _run(["g++", "-O2", "-std=c++17", "-o", gen,
          os.path.join(CSRC, "gen.cpp"), os.path.join(CSRC, "builder.cpp")], verbose)
    tmp = os.path.join(BUILD, "generated.tmp")
    shutil.rmtree(tmp, ignore_errors=True)
    os.makedirs(tmp)
    _run([gen, tmp, *(layouts_from_env() if extra is None else extra)], verbose)
    units = open(os.path.join(tmp, "units.txt")).read().split()
    # replace the generated directory's contents (unchanged files keep their times)
    keep = set(os.listdir(tmp))
    for f in os.listdir(GEN):
        if f not in keep:
            os.remove(os.path.join(GEN, f))
    for f in keep:
        src, dst = os.path.join(tmp, f), os.path.join(GEN, f)
        if not os.path.exists(dst) or open(dst, "rb").read() != open(src, "rb").read():
            shutil.copyfile(src, dst)
    shutil.rmtree(tmp, ignore_errors=True)
    return units


def build(verbose: bool = True, extra=None) -> str:
    units = generate(verbose, extra)
    objdir = os.path.join(BUILD, "obj")
    os.makedirs(objdir, exist_ok=True)
    sources = [os.path.join(CSRC, "e3mi.hip"), os.path.join(CSRC, "convr.hip"),
               os.path.join(CSRC, "builder.cpp")] + \
              [os.path.join(GEN, u) for u in units]
    objs = []
    cmds = []
    for src in sources:
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        objs.append(obj)
        cmds.append([HIPCC, *HIP_FLAGS, "-c", "-o", obj, src])
    with cf.ThreadPoolExecutor(max_workers=_jobs()) as ex:
        for fut in [ex.submit(_run, c, verbose) for c in cmds]:
            fut.result()
    out_tmp = LIB + ".tmp"
    _run([HIPCC, *HIP_FLAGS, "-shared", "-o", out_tmp, *objs], verbose)
    os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
