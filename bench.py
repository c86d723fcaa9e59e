"""Benchmark: fused channelwise CG convolution, forward + backward, on one MI355X.

One step = conv forward + conv backward (harmonics, per-edge coefficient
pre-contraction, channelwise contraction with path weights, receiver-segment
reduction; backward edge sweep, sender-segment dx reduction, dvec) over the
24,000-atom synthetic water box (8,000 rigid H2O, periodic, r_c = 5 A),
x = 128x0e+128x1o+128x2e+128x3o, harmonics l <= 3, outputs l <= 3, fp32.
Inputs are resident in HBM before the timed region.  The CSR graph build is
timed separately (graph_build_ms); the standalone weighted tensor product
(200,000 rows, 128x0e+128x1o+128x2e) is reported under "tp".

Prints ONE JSON line.  Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402

METRIC = "edges/sec conv fwd+bwd (fp32, lmax=3, 128ch) + achieved HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0
# fp32 vector peak without packed math: 256 CUs x 4 SIMDs x 16 lanes x 2 flop (FMA) x 2.4 GHz.
# The kernels are built with packed fp32 disabled, so this is the attainable VALU peak;
# the published 157.3 TFLOP/s counts the packed FMA.
VALU_PEAK_TFLOPS = 78.6
VALU_PEAK_PACKED_TFLOPS = 157.3


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def conv_bytes(N, E, C, D_in, D_out, P):
    """Algorithmic bytes (inputs + outputs, no scratch) per kernel, and totals."""
    f = 4
    idx_fwd = E * 4 * 2 + (N + 1) * 4          # edge id + sender per receiver-CSR slot, rowptr
    k = {}
    k["conv_fwd"] = N * D_in * C * f + E * 3 * f + E * P * C * f + N * D_out * C * f + idx_fwd
    # backward sweep: reads x, vec, s, dm, indices; writes ds (+ scratch, not counted)
    k["conv_bwd_edges"] = (N * D_in * C * f + E * 3 * f + E * P * C * f + N * D_out * C * f
                           + E * P * C * f + E * 4 * 3 + (N + 1) * 4)
    k["conv_bwd_dx"] = N * D_in * C * f + (N + 1) * 4
    k["conv_bwd_dvec"] = E * 3 * f * 2 + E * 4
    fwd = k["conv_fwd"]
    bwd = (N * D_in * C * f + E * 3 * f + E * P * C * f + N * D_out * C * f      # inputs
           + N * D_in * C * f + E * 3 * f + E * P * C * f + E * 4 * 3 + (N + 1) * 4 * 2)  # outputs + idx
    return k, fwd, bwd


def radial_bytes(N, E, C, D_in, D_out, P, K):
    """Algorithmic bytes of the convolution with fused radial weights (h [E, K]
    and W [K, P, C] replace s); ds is scratch, not counted."""
    f = 4
    fwd = (N * D_in * C * f + E * 3 * f + E * K * f + K * P * C * f + N * D_out * C * f
           + E * 4 * 2 + (N + 1) * 4)
    bwd = (N * D_in * C * f + E * 3 * f + E * K * f + K * P * C * f + N * D_out * C * f   # inputs
           + N * D_in * C * f + E * 3 * f + E * K * f + K * P * C * f                      # outputs
           + E * 4 * 3 + (N + 1) * 4 * 2)
    return fwd, bwd


KERNEL_SOURCES = ["paper_2609_35099_amd/csrc/e3mi.hip", "paper_2609_35099_amd/csrc/e3mi_impl.h",
                  "paper_2609_35099_amd/csrc/convr.hip", "paper_2609_35099_amd/csrc/gen.cpp",
                  "paper_2609_35099_amd/csrc/builder.cpp", "paper_2609_35099_amd/csrc/builder.h"]
COUNTERS = os.path.join(ROOT, "profiles", "conv_water8k_tp200k_hbm_bytes.txt")


def source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()[:16]


UTIL = os.path.join(ROOT, "profiles", "util_water8k_tp200k.txt")


def counter_util(kernel: str, metric: str):
    """A per-kernel utilisation figure (percent) from the committed rocprofv3
    summary, or None if missing or taken on a different kernel source."""
    try:
        lines = open(UTIL).read().splitlines()
    except OSError:
        return None
    want = source_hash()
    for ln in lines:
        p = ln.split()
        if len(p) == 5 and p[0] == "util" and p[1] == kernel and p[2] == metric and p[3] == want:
            return float(p[4])
    return None


def fma_counts(plan):
    """FMA-equivalent VALU operations per edge and channel of the forward and
    backward sweeps, counted as the kernel generator counts them.

    Forward: one per (output, x) pre-contraction entry plus the path-weight
    product per output row.  Backward, per path, the cheapest of three orders
    of the same sums (the one the generated code uses), each with two per
    harmonic row (ds = y . B and dy += s B):
      A: two per entry (dm x product, x cotangent), one per coupling
         coefficient, plus min(d1, d3) for the path weight;
      B: one per entry, one per coefficient, one per (M, m2) pair, min(d1, d3);
      C: one per coefficient, two per (m1, m2) pair, d1;
    and the paths whose coupling is the identity between the output block and
    the x block or the harmonic block (the (0, l, l) and (l, 0, l) paths) take
    2 d3 + 3 in all."""
    i0, i1, i2, val = plan.records()
    paths = plan.paths()
    pairs = len(set(zip(i0.tolist(), i1.tolist())))
    bwd = 0
    for (l1, l2, l3, _, x_off, y_off, out_off) in paths.tolist():
        d1, d2, d3 = 2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1
        sel = (i0 >= out_off) & (i0 < out_off + d3) & (i1 >= x_off) & (i1 < x_off + d1) \
            & (i2 >= y_off) & (i2 < y_off + d2)
        a, b, c = i0[sel].tolist(), i1[sel].tolist(), i2[sel].tolist()
        nnz, nE = len(a), len(set(zip(a, b)))
        nMm2, nm1m2 = len(set(zip(a, c))), len(set(zip(b, c)))
        v = val[sel]
        unit = nE == d3 and nnz == nE and bool(np.all(np.abs(v - 1.0) <= 1e-12))
        if unit and ((d1 == 1 and len(set(c)) == d3) or (d2 == 1 and len(set(b)) == d3)):
            bwd += 2 * d3 + 3  # identity coupling with the x or the harmonic block
            continue
        bwd += min(2 * nE + nnz + min(d1, d3), nE + nnz + nMm2 + min(d1, d3), nnz + 2 * nm1m2 + d1) + 2 * d2
    return pairs + plan.D_out, bwd


def counter_traffic(kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None
    if it is missing or was taken on a different kernel source."""
    try:
        lines = open(COUNTERS).read().splitlines()
    except OSError:
        return None
    want = source_hash()
    for ln in lines:
        p = ln.split()
        if len(p) == 4 and p[0] == "traffic" and p[1] == kernel and p[2] == want:
            return int(p[3])
    return None


def step_counter_bytes(kernels):
    """Sum of the committed counter bytes of the convolution step's kernels
    (None if any is missing or stale)."""
    tot = 0
    for k in ("conv_fwd", "conv_bwd_edges", "conv_bwd_dx", "conv_bwd_dvec"):
        if k not in kernels:
            continue
        t = counter_traffic(k)
        if t is None:
            return None
        tot += t
    return tot


def tp_bytes(R, C, D_in, D_sh, D_out, P):
    return R * (D_in * C + D_sh + P * C + D_out * C) * 4


def tp_bwd_bytes(R, C, D_in, D_sh, D_out, P):
    """x, y, w, dz read; dx, dy, dw written."""
    return R * (2 * D_in * C + 2 * D_sh + 2 * P * C + D_out * C) * 4


# The paper's e3j numbers for its channel sweep on an H100 (GB/s, channels 64..1024;
# None where the kernel does not run).  Context only: other hardware, other graphs.
PAPER_H100_GBPS = {
    "lmax2": {"fwd_cuda": [625, 955, 913, 956, 880], "fwd_pallas": [None, 1621, 1669, 1716, 1871],
              "bwd_cuda": [446, 709, 638, 560, 623], "bwd_pallas": [None, 1267, 1292, 1319, 1328]},
    "lmax3": {"fwd_cuda": [389, 569, 573, 562, 538], "fwd_pallas": [None, 1818, 1859, 2074, 2067],
              "bwd_cuda": [310, 423, 402, 317, 183], "bwd_pallas": [None, 1407, 1432, 1483, 1599]},
}


def sweep(args, dev):
    """Forward and backward throughput (GB/s of inputs + outputs, the paper's
    definition) over C = 64..1024 with N*C = 2^22 (l_max 2) or 2^21 (l_max 3)."""
    import torch
    from paper_2609_35099_amd import e3mi
    rows = []
    for lmax in (2, 3):
        for C in (64, 128, 256, 512, 1024):
            scfg = synth.sweep_config(lmax, C)
            g = synth.graph(scfg)
            N, E = g.n_nodes, g.sender.shape[0]
            plan = e3mi.Plan(scfg.irreps, scfg.lmax_sh, scfg.lmax_out)
            G = e3mi.Graph(torch.from_numpy(g.sender).to(dev), torch.from_numpy(g.receiver).to(dev), N)
            x = synth.normal_device(scfg.cid, 1, (N, plan.D_in, C), dev)
            s = synth.normal_device(scfg.cid, 2, (E, plan.P, C), dev)
            dm = synth.normal_device(scfg.cid, 3, (N, plan.D_out, C), dev)
            vs = torch.from_numpy(g.vec).to(dev)
            m = torch.empty((N, plan.D_out, C), dtype=torch.float32, device=dev)
            dx = torch.empty_like(x)
            dvec = torch.empty_like(vs)
            ds = torch.empty_like(s)
            ws = e3mi.workspace(e3mi.conv_workspace_size(plan, G)[1])
            for _ in range(2):
                e3mi.conv_fwd(plan, G, x, vs, s, out=m)
                e3mi.conv_bwd(plan, G, x, vs, s, dm, dx=dx, dvec=dvec, ds=ds, ws=ws)
            torch.cuda.synchronize()
            f0, f1, b1 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            tf = tb = 0.0
            for _ in range(5):
                f0.record()
                e3mi.conv_fwd(plan, G, x, vs, s, out=m)
                f1.record()
                e3mi.conv_bwd(plan, G, x, vs, s, dm, dx=dx, dvec=dvec, ds=ds, ws=ws)
                b1.record()
                torch.cuda.synchronize()
                tf += f0.elapsed_time(f1) / 5
                tb += f1.elapsed_time(b1) / 5
            _, fb, bb = conv_bytes(N, E, C, plan.D_in, plan.D_out, plan.P)
            rows.append({"lmax": lmax, "channels": C, "n_nodes": N, "n_edges": E,
                         "avg_neighbours": round(E / N, 1), "fwd_ms": round(tf, 4), "bwd_ms": round(tb, 4),
                         "fwd_GBps": round(fb / (tf * 1e-3) / 1e9, 1), "bwd_GBps": round(bb / (tb * 1e-3) / 1e9, 1)})
            log(f"sweep l_max {lmax} C {C}: N {N} E {E}: fwd {rows[-1]['fwd_GBps']} GB/s, "
                f"bwd {rows[-1]['bwd_GBps']} GB/s")
            del x, s, dm, m, dx, dvec, ds, ws, G
            torch.cuda.empty_cache()
    return {"definition": "GB/s = (inputs + outputs) / time, per pass; water boxes with ~45 neighbours; "
                          "N*C = 2^22 at l_max 2, 2^21 at l_max 3; x = C x (0e+1o+..); N(0,1) weights",
            "rows": rows, "paper_h100_GBps_context": PAPER_H100_GBPS}


# Streaming probes of the library (e3_probe_stream): the bandwidth HBM sustains
# for a read:write mix, with the sweeps' own load/store instructions.  Each
# entry: name, read units, write units per step, bytes per lane, flags (1: non-
# temporal loads, 2: non-temporal stores), and the kernels whose counter traffic
# has that mix and instruction width (their ceiling).
CEILING_PROBES = [
    ("read_nt_b128", 16, 0, 16, 1, ["conv_bwd_dx"]),   # the dx segment sum reads T (98% reads)
    ("read_nt_b64", 16, 0, 8, 1, []),
    ("read_nt_b32", 16, 0, 4, 1, []),
    ("read_b128", 16, 0, 16, 0, []),
    ("write_nt_b128", 0, 16, 16, 2, []),
    ("write_b128", 0, 16, 16, 0, []),
    ("copy_nt_b128", 8, 8, 16, 3, []),
    ("mix_14r1w_b64", 14, 1, 8, 3, ["conv_fwd"]),       # forward sweep: 93:7 by its counters, 8 bytes per lane
    ("mix_14r16w_b32", 14, 16, 4, 3, ["conv_bwd_edges"]),  # backward sweep: 47:53, 4 bytes per lane
    ("mix_2r6w_b64", 2, 6, 8, 3, ["tp_fwd"]),           # tensor product: 24:76
    ("mix_8r2w_b64", 8, 2, 8, 3, ["tp_bwd"]),           # tensor-product backward: 81:19
]


def hbm_ceilings(dev, reps=10, gib=6):
    """Run every streaming probe over `gib` GiB buffers: {name: GB/s and the mix}."""
    import torch
    from paper_2609_35099_amd import e3mi
    n = (gib << 30) // 4
    src = torch.zeros(n, dtype=torch.float32, device=dev)
    dst = torch.empty(n, dtype=torch.float32, device=dev)
    res = {}
    for name, ru, wu, width, flags, _ in CEILING_PROBES:
        for _ in range(2):
            e3mi.probe_stream(src if ru else None, dst if wu else None, ru, wu, width, flags)
        torch.cuda.synchronize()
        e3mi.timing_reset()
        e3mi.timing_enable(True)
        for _ in range(reps):
            br, bw = e3mi.probe_stream(src if ru else None, dst if wu else None, ru, wu, width, flags)
        torch.cuda.synchronize()
        e3mi.timing_enable(False)
        ms_tot, cnt = e3mi.timing_read()["probe_stream"]
        ms = ms_tot / cnt
        res[name] = {"GBps": round((br + bw) / (ms * 1e-3) / 1e9, 1), "ms": round(ms, 4),
                     "read_bytes": br, "write_bytes": bw, "bytes_per_lane": width,
                     "nt_loads": bool(flags & 1), "nt_stores": bool(flags & 2)}
        log(f"ceiling {name}: {res[name]['GBps']} GB/s")
    del src, dst
    torch.cuda.empty_cache()
    return res


def against_ceilings(kernels, ceil):
    """Counter GB/s of each kernel with committed counter bytes, as a fraction of
    the probe that matches its read:write mix."""
    for name, _, _, _, _, users in CEILING_PROBES:
        for k in users:
            if k not in kernels or name not in ceil:
                continue
            t = counter_traffic(k)
            if t is None:
                continue
            gbps = t / (kernels[k]["ms"] * 1e-3) / 1e9
            kernels[k].update({"counter_GBps": round(gbps, 1), "ceiling": name,
                               "frac_of_ceiling": round(gbps / ceil[name]["GBps"], 4)})


# ---------------------------------------------------------------- profile summaries
# rocprofv3 runs behind the files in profiles/ (on an MI355X machine, after
# `cd /tmp && export TMPDIR=/tmp`; $REPO is the repository root, $OUT a results
# directory): a kernel trace per bench section, one HBM byte counter per run,
# and the utilisation counters.  `python bench.py --summarize-profiles $OUT`
# reduces their CSV output to the committed summaries.
PROF_TRACE = ("rocprofv3 --kernel-trace --stats --output-format csv -d $OUT/trace_{s} -o trace "
              "-- python -u $REPO/bench.py --only {s} --steps 10 --warmup 2 --no-cpu-baseline")
PROF_PMC = ("rocprofv3 --pmc {c} --output-format csv -d $OUT/pmc_{s}_{c} -o p "
            "-- python -u $REPO/bench.py --only {s} --steps 2 --warmup 1 --no-cpu-baseline --copy-probe")
PROF_UTIL = ("rocprofv3 --pmc MfmaUtil VALUBusy LdsUtil SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_INSTS_VALU --output-format csv "
             "-d $OUT/util_{s} -o u -- python -u $REPO/bench.py --only {s} --steps 2 --warmup 1 --no-cpu-baseline")
PROF_FILES = [  # file, kind, sections, title
    ("conv_water8k_tp200k_kernel_trace.txt", "trace", ["conv", "tp"],
     "Kernel-time summary: convolution forward+backward (24,000-atom water box, 128 ch, l<=3) and weighted TP "
     "forward+backward (200,000 rows)"),
    ("bwd2_water8k_kernel_trace.txt", "trace", ["bwd2"],
     "Kernel-time summary: double backward of the convolution (same water box)"),
    ("generic_water8k_kernel_trace.txt", "trace", ["generic"],
     "Kernel-time summary: the convolution step (same water box) on the composed path (kind_*: generated "
     "single-block kernels, block by block) and on the runtime-record path (convr_*)"),
    ("linear_water8k_kernel_trace.txt", "trace", ["linear"],
     "Kernel-time summary: linear mixing of the convolution output (24,000 nodes, 34 path blocks -> 8 irreps, 128 ch)"),
    ("radial_water8k_kernel_trace.txt", "trace", ["radial"],
     "Kernel-time summary: convolution with fused radial weights (same water box, K = 8 Bessel features)"),
    ("conv_water8k_tp200k_hbm_bytes.txt", "hbm", ["conv", "tp"],
     "HBM byte counters per dispatch (FETCH_SIZE, WRITE_SIZE in KiB), scaled by a plain 2 GiB device copy; "
     "one counter per run"),
    ("radial_water8k_hbm_bytes.txt", "hbm", ["radial"],
     "HBM byte counters per dispatch (FETCH_SIZE, WRITE_SIZE in KiB), scaled by a plain 2 GiB device copy; "
     "one counter per run"),
    ("util_water8k_tp200k.txt", "util", ["conv", "linear", "radial", "tp", "bwd2", "generic"],
     "Per-kernel utilisation (rocprofv3 derived metrics, per dispatch, mean over dispatches)"),
]
# kernel symbol -> short name used by the library's timing and the summaries
PROF_NAMES = [("k_conv_bwd_edges", "conv_bwd_edges"), ("k_conv_bwd3", "conv_bwd3"), ("k_conv_fwd3", "conv_fwd3"),
              ("k_conv_fwd_rad", "conv_fwd_rad"), ("k_conv_bwd_rad", "conv_bwd_rad_edges"),
              ("k_conv_fwd", "conv_fwd"), ("k_conv_bwd_dx", "conv_bwd_dx"), ("k_conv_bwd_dvec", "conv_bwd_dvec"),
              ("k_conv_bwd_dy", "conv_bwd_dy"), ("k_zero_pad", "zero_pad"), ("k_rad_grad", "rad_grad"),
              ("k_rad_dw_sum", "rad_dw_sum"), ("k_rad_dh_sum", "rad_dh_sum"), ("k_lin_gemm", "linear_gemm(fwd+dx)"),
              ("k_lin_dw_sum", "linear_dw_sum"), ("k_lin_dw", "linear_dw"), ("k_lin_transpose", "linear_transpose"),
              ("k_tp_bwd_dy", "tp_bwd_dy"), ("k_tp_bwd", "tp_bwd"), ("k_tpg_sum", "tp_records_sum"),
              ("k_tpg", "tp_records"), ("k_tp", "tp_fwd"), ("k_sh_bwd", "sh_bwd"), ("k_sh", "sh"),
              ("k_graph_keys", "graph_keys"), ("k_graph_rowptr", "graph_rowptr"), ("k_graph_finish", "graph_finish"),
              ("k_graph_r2s", "graph_r2s"), ("k_probe", "probe_stream"), ("k_convr_fwd", "convr_fwd"),
              ("k_convr_bwd", "convr_bwd"), ("k_convr_dvec", "convr_dvec"), ("k_convr_dy", "convr_dy"),
              ("k_zero_rows", "zero_rows")]
COPY_PROBE = "copy_probe(__amd_rocclr_copyBuffer)"


def _prof_short(name, cache={}):
    import re
    import subprocess
    if name not in cache:
        d = name
        if name.startswith("_Z"):
            d = subprocess.run(["c++filt", name], capture_output=True, text=True).stdout.strip() or name
        short = None
        if "__amd_rocclr_copyBuffer" in d:
            short = COPY_PROBE
        else:
            for sym, nm in PROF_NAMES:
                if re.search(r"(?<![A-Za-z0-9_])" + sym + r"(?=[<(]|$)", d):
                    short = nm
                    break
            if short and "e3gen::K_" in d:  # a single-block kind of the composed path
                short = "kind_" + short
        cache[name] = short
    return cache[name]


def _prof_rows(root, pattern):
    import csv
    import glob
    out = []
    for f in glob.glob(os.path.join(root, pattern), recursive=True):
        out += list(csv.DictReader(open(f)))
    return out


def _prof_trace(root, sec):
    d, tot = {}, 0.0
    for r in _prof_rows(root, f"trace_{sec}/**/*kernel_trace.csv"):
        dt = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6
        tot += dt
        k = _prof_short(r["Kernel_Name"])
        if k is not None:
            d.setdefault(k, []).append(dt)
    lines = [f"## section {sec}"]
    for k, v in sorted(d.items(), key=lambda kv: -sum(kv[1])):
        lines.append(f"{k:<36s} {len(v):5d} {sum(v) / len(v):9.4f} {min(v):9.4f} {max(v):9.4f} "
                     f"{100 * sum(v) / tot:6.2f}%")
    return lines


def _prof_counter(root, sec, ctr, rows_glob):
    d = {}
    rs = _prof_rows(root, rows_glob)
    copies = [int(r["Grid_Size"]) for r in rs if "copyBuffer" in r["Kernel_Name"]]
    big = max(copies) if copies else -1
    for r in rs:
        if r["Counter_Name"] != ctr:
            continue
        k = _prof_short(r["Kernel_Name"])
        if k is None or (k == COPY_PROBE and int(r["Grid_Size"]) != big):
            continue  # small runtime copies are not the 2 GiB calibration copy
        slot = d.setdefault(k, {})
        slot[r.get("Dispatch_Id")] = slot.get(r.get("Dispatch_Id"), 0.0) + float(r["Counter_Value"])
    return {k: sum(v.values()) / len(v) for k, v in d.items()}


def _prof_hbm(root, sec, h):
    f = _prof_counter(root, sec, "FETCH_SIZE", f"pmc_{sec}_FETCH_SIZE/**/*counter_collection.csv")
    w = _prof_counter(root, sec, "WRITE_SIZE", f"pmc_{sec}_WRITE_SIZE/**/*counter_collection.csv")
    # scale: the counter bytes a plain copy of exactly 2 GiB each way reports
    rs_, ws_ = 2097152.0 / f[COPY_PROBE], 2097152.0 / w[COPY_PROBE]
    lines = [f"## section {sec}: the 2 GiB copy reads FETCH_SIZE {f[COPY_PROBE]:.1f} KiB -> read scale {rs_:.4f}; "
             f"WRITE_SIZE {w[COPY_PROBE]:.1f} KiB -> write scale {ws_:.4f}",
             "# kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | read bytes | write bytes | total bytes (scaled)"]
    for k in sorted(f):
        if k == COPY_PROBE or k not in w:
            continue
        rb, wb = int(f[k] * 1024 * rs_), int(w[k] * 1024 * ws_)
        lines.append(f"{k:<24s} {f[k]:14.1f} {w[k]:14.1f} {rb:14d} {wb:14d} {rb + wb:14d}")
        lines.append(f"traffic {k} {h} {rb + wb}")
    return lines


def _prof_util(root, sec, h):
    mets = ["MfmaUtil", "VALUBusy", "LdsUtil", "SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_INSTS_VALU"]
    d = {}
    for r in _prof_rows(root, f"util_{sec}/**/*counter_collection.csv"):
        k = _prof_short(r["Kernel_Name"])
        if k is None or r["Counter_Name"] not in mets:
            continue
        slot = d.setdefault(k, {}).setdefault(r["Counter_Name"], {})
        slot[r.get("Dispatch_Id")] = slot.get(r.get("Dispatch_Id"), 0.0) + float(r["Counter_Value"])
    lines = [f"## section {sec}"]
    for k in sorted(d, key=lambda k: -sum(d[k].get("SQ_INSTS_VALU", {0: 0}).values())):
        m = {n: sum(v.values()) / len(v) for n, v in d[k].items()}
        lines.append(f"{k:<24s} {m.get('MfmaUtil', 0):8.2f} {m.get('VALUBusy', 0):7.2f} {m.get('LdsUtil', 0):7.2f} "
                     f"{m.get('SQ_INSTS_VALU_MFMA_MOPS_F32', 0):14.0f} {m.get('SQ_INSTS_VALU', 0):14.0f}")
        for n in ("MfmaUtil", "VALUBusy", "LdsUtil"):
            lines.append(f"util {k} {n} {h} {m.get(n, 0):.2f}")
    return lines


def summarize_profiles(root, only=None):
    """Write the profiles/ summaries from rocprofv3 CSV output under root,
    tagged with the hash of the kernel sources in this tree."""
    h = source_hash()
    for fname, kind, secs, title in PROF_FILES:
        if only and fname not in only:
            continue
        if kind == "trace":
            cmds = [PROF_TRACE.format(s=s) for s in secs]
            body = ["# columns: kernel | calls | avg ms | min ms | max ms | share of the run's GPU time"]
            for sec in secs:
                body += _prof_trace(root, sec)
        elif kind == "hbm":
            cmds = [PROF_PMC.format(s=s, c=c) for s in secs for c in ("FETCH_SIZE", "WRITE_SIZE")]
            body = []
            for sec in secs:
                body += _prof_hbm(root, sec, h)
        else:
            cmds = [PROF_UTIL.format(s=s) for s in secs]
            body = ["# MfmaUtil, VALUBusy, LdsUtil in percent of the kernel's duration; MOPS_F32 in units of "
                    "512 flop", "# kernel | MfmaUtil | VALUBusy | LdsUtil | SQ_INSTS_VALU_MFMA_MOPS_F32 | "
                    "SQ_INSTS_VALU"]
            for sec in secs:
                body += _prof_util(root, sec, h)
        head = [f"# {title}", f"# source hash (e3mi.hip, e3mi_impl.h, convr.hip, gen.cpp, builder.*): {h}",
                "# on an MI355X machine, after `cd /tmp && export TMPDIR=/tmp`, with $REPO the repository root and "
                "$OUT a results directory:"] + ["#   " + c for c in cmds]
        with open(os.path.join(ROOT, "profiles", fname), "w") as fh:
            fh.write("\n".join(head + body) + "\n")
        log(f"wrote profiles/{fname}")


def cpu_model() -> str:
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def cpu_baseline(cfg, g, x, dm, seconds=12.0):
    """The fp64 oracle on the host cores, on a bounded sample of the same workload:
    forward for sampled receivers and backward for sampled senders and edges."""
    import torch
    from oracle import conv as oconv
    from oracle import irreps as oirreps
    lay = oirreps.layout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    rng = np.random.default_rng(123)
    W = synth.bessel_matrix(cfg)
    edges_done, t_used, n_batches = 0, 0.0, 0
    def compact(sel):
        # the sub-problem on the nodes these edges touch, renumbered 0..k-1
        nodes, inv = np.unique(np.concatenate([g.sender[sel], g.receiver[sel]]), return_inverse=True)
        k = sel.shape[0]
        return nodes, inv[:k].astype(np.int32), inv[k:].astype(np.int32)

    while t_used < seconds and n_batches < 256:
        b = rng.choice(g.n_nodes, 4, replace=False)
        sel_r = np.nonzero(np.isin(g.receiver, b))[0]
        sel_s = np.nonzero(np.isin(g.sender, b))[0]
        s_r = synth.edge_weights_rows(cfg, g.vec, sel_r, W=W)
        s_s = synth.edge_weights_rows(cfg, g.vec, sel_s, W=W)
        nr, snd_r, rcv_r = compact(sel_r)
        ns, snd_s, rcv_s = compact(sel_s)
        br = np.searchsorted(nr, b)
        bs = np.searchsorted(ns, b)
        xr, xs_, dms_ = x[nr], x[ns], dm[ns]
        t0 = time.perf_counter()
        oconv.conv_fwd(lay, xr, g.vec[sel_r], s_r, snd_r, rcv_r, nr.shape[0], receivers=br)
        oconv.conv_bwd(lay, xs_, g.vec[sel_s], s_s, dms_, snd_s, rcv_s, ns.shape[0], senders=bs)
        t_used += time.perf_counter() - t0
        edges_done += (sel_r.shape[0] + sel_s.shape[0]) / 2.0
        n_batches += 1
    return {"value": edges_done / t_used, "unit": "edges/s", "cores": len(os.sched_getaffinity(0)),
            "kind": "oracle", "rate": "extrapolated from the sample",
            "sample": f"{n_batches} batches of 4 random atoms: forward of their {int(edges_done)} in-edges "
                      f"(avg of in/out counts) and full backward (dx of the atoms, ds/dvec of their "
                      f"out-edges), float64, {t_used:.1f} s; rate = edges / (t_fwd + t_bwd), extrapolated "
                      f"to the whole workload",
            "cpu": cpu_model(), "numpy": np.__version__, "torch_threads": torch.get_num_threads(),
            "affinity_cores": len(os.sched_getaffinity(0))}


def oracle_configs():
    """The fp64 oracle on whole workloads of the three small configurations, on
    the host cores (a reported baseline): convolution forward + backward of the
    64-atom cube and the 1,000-molecule water box, and the weighted tensor
    product of 200,000 rows (in chunks of 8,192 rows).  Best of three where one
    run takes under 30 s, else one run."""
    import torch
    from oracle import conv as oconv
    from oracle import irreps as oirreps
    from oracle import sh as osh
    from oracle import tp as otp
    res = {}

    def timed(fn):
        best, n = float("inf"), 0
        while n < 3:
            t0 = time.perf_counter()
            fn()
            dt = time.perf_counter() - t0
            best, n = min(best, dt), n + 1
            if dt >= 30.0:
                break
        return best, n

    for name in ("cube64", "water1k"):
        cfg = synth.CONFIGS[name]
        g = synth.graph(cfg)
        lay = oirreps.layout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
        E = int(g.sender.shape[0])
        x = synth.node_features(cfg, g.n_nodes)
        s = synth.edge_weights(cfg, g.vec, 0, E)
        dm = synth.out_cotangent(cfg, g.n_nodes)
        tf, nf = timed(lambda: oconv.conv_fwd(lay, x, g.vec, s, g.sender, g.receiver, g.n_nodes))
        tb, nb = timed(lambda: oconv.conv_bwd(lay, x, g.vec, s, dm, g.sender, g.receiver, g.n_nodes))
        res[name] = {"edges": E, "fwd_s": round(tf, 3), "bwd_s": round(tb, 3), "runs": [nf, nb],
                     "edges_per_s": round(E / (tf + tb), 1)}
        log(f"oracle {name}: {res[name]}")
    cfg = synth.CONFIGS["tp200k"]
    lay = oirreps.layout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    x, u, w = synth.tp_inputs(cfg)
    y = osh.sh_unit(cfg.lmax_sh, u.astype(np.float64))
    R, chunk = x.shape[0], 8192

    def tp_all():
        for r0 in range(0, R, chunk):
            otp.tp(lay, x[r0:r0 + chunk], y[r0:r0 + chunk], w[r0:r0 + chunk])

    tt, nt = timed(tp_all)
    res["tp200k"] = {"rows": R, "fwd_s": round(tt, 3), "runs": nt, "rows_per_s": round(R / tt, 1)}
    log(f"oracle tp200k: {res['tp200k']}")
    return {"kind": "oracle", "dtype": "f64", "configs": res, "cpu": cpu_model(), "numpy": np.__version__,
            "torch_threads": torch.get_num_threads(), "affinity_cores": len(os.sched_getaffinity(0)),
            "blas_env": {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS",
                                                        "MKL_NUM_THREADS") if os.environ.get(k)}}


def capacity(args, dev):
    """The capacity workload: 70,000 H2O (210,000 atoms, about 11M edges) at 64
    channels, forward + backward on one GPU with every operand resident (s and
    ds alone are about 97 GB each)."""
    import torch
    from paper_2609_35099_amd import e3mi
    cfg = synth.CONFIGS["water70k"]
    t0 = time.perf_counter()
    g = synth.graph(cfg)
    plan = e3mi.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    N, E, C = g.n_nodes, int(g.sender.shape[0]), cfg.channels
    xs = torch.from_numpy(synth.node_features(cfg, N)).to(dev)
    vs = torch.from_numpy(g.vec).to(dev)
    s = synth.normal_device(cfg.cid, 2, (E, plan.P, C), dev)
    dms = synth.normal_device(cfg.cid, 3, (N, plan.D_out, C), dev)
    graph = e3mi.Graph(torch.from_numpy(g.sender).to(dev), torch.from_numpy(g.receiver).to(dev), N)
    log(f"capacity inputs ready: N={N} E={E} ({time.perf_counter() - t0:.1f} s)")
    m = torch.empty((N, plan.D_out, C), dtype=torch.float32, device=dev)
    dx = torch.empty((N, plan.D_in, C), dtype=torch.float32, device=dev)
    dvec = torch.empty((E, 3), dtype=torch.float32, device=dev)
    ds = torch.empty((E, plan.P, C), dtype=torch.float32, device=dev)
    ws = e3mi.workspace(e3mi.conv_workspace_size(plan, graph)[1])

    def step():
        e3mi.conv_fwd(plan, graph, xs, vs, s, out=m)
        e3mi.conv_bwd(plan, graph, xs, vs, s, dms, dx=dx, dvec=dvec, ds=ds, ws=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e3mi.timing_reset()
    e3mi.timing_enable(True)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    e3mi.timing_enable(False)
    per = e3mi.timing_read()
    ms_step = ev0.elapsed_time(ev1) / args.steps
    _, fwd_b, bwd_b = conv_bytes(N, E, C, plan.D_in, plan.D_out, plan.P)
    res = {"workload": "water box, 70,000 rigid H2O = 210,000 atoms, periodic, r_c 5 A; x 64x0e+64x1o+64x2e+64x3o, "
                       "harmonics l<=3, outputs l<=3, forward + backward convolution",
           "n_nodes": N, "n_edges": E, "channels": C, "ms_per_step": round(ms_step, 3),
           "edges_per_s": E / (ms_step * 1e-3),
           "step_alg_GBps": round((fwd_b + bwd_b) / (ms_step * 1e-3) / 1e9, 1),
           "step_alg_frac": round((fwd_b + bwd_b) / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "kernels": {k: {"ms": round(v[0] / v[1], 4), "launches": v[1]} for k, v in per.items()},
           "device_memory_GB": round(torch.cuda.max_memory_allocated(dev) / 1e9, 1)}
    log(f"capacity: {ms_step:.3f} ms/step, {E / ms_step / 1e3:.1f} M edges/s")
    del m, dx, dvec, ds, ws, s, dms, graph, xs, vs
    torch.cuda.empty_cache()
    return res


def oracle_config4(part="both", chunk_nodes=2048):
    """The fp64 oracle on the whole 24,000-atom water box, once, in node chunks
    (a reported baseline): the forward by chunks of receivers (their in-edges),
    the backward by chunks of senders (dx of the senders, ds and dvec of their
    out-edges, so every edge once).  Each chunk runs on the sub-problem of the
    nodes its edges touch; only the oracle calls are timed (the chunk's edge
    weights are generated outside the timed region)."""
    import torch
    from oracle import conv as oconv
    from oracle import irreps as oirreps
    cfg = synth.CONFIGS["water8k"]
    g = synth.graph(cfg)
    lay = oirreps.layout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    x = synth.node_features(cfg, g.n_nodes)
    dm = synth.out_cotangent(cfg, g.n_nodes)
    W = synth.bessel_matrix(cfg)
    N, E = g.n_nodes, int(g.sender.shape[0])
    by_r = np.argsort(g.receiver, kind="stable")
    by_s = np.argsort(g.sender, kind="stable")
    ptr_r = np.searchsorted(g.receiver[by_r], np.arange(N + 1))
    ptr_s = np.searchsorted(g.sender[by_s], np.arange(N + 1))

    def compact(sel):
        nodes, inv = np.unique(np.concatenate([g.sender[sel], g.receiver[sel]]), return_inverse=True)
        k = sel.shape[0]
        return nodes, inv[:k].astype(np.int32), inv[k:].astype(np.int32)

    t_f = t_b = 0.0
    done_f = done_b = 0
    for c0 in range(0, N if part in ("both", "fwd") else 0, chunk_nodes):
        c1 = min(N, c0 + chunk_nodes)
        sel = by_r[ptr_r[c0]:ptr_r[c1]]
        s_sel = synth.edge_weights_rows(cfg, g.vec, sel, W=W)
        nodes, snd, rcv = compact(sel)
        rows = np.searchsorted(nodes, np.arange(c0, c1))
        t0 = time.perf_counter()
        oconv.conv_fwd(lay, x[nodes], g.vec[sel], s_sel, snd, rcv, nodes.shape[0], receivers=rows)
        t_f += time.perf_counter() - t0
        done_f += sel.shape[0]
        log(f"oracle water8k forward: receivers {c1}/{N}, {done_f} edges, {t_f:.0f} s")
    for c0 in range(0, N if part in ("both", "bwd") else 0, chunk_nodes):
        c1 = min(N, c0 + chunk_nodes)
        sel = by_s[ptr_s[c0]:ptr_s[c1]]
        s_sel = synth.edge_weights_rows(cfg, g.vec, sel, W=W)
        nodes, snd, rcv = compact(sel)
        rows = np.searchsorted(nodes, np.arange(c0, c1))
        t0 = time.perf_counter()
        oconv.conv_bwd(lay, x[nodes], g.vec[sel], s_sel, dm[nodes], snd, rcv, nodes.shape[0], senders=rows)
        t_b += time.perf_counter() - t0
        done_b += sel.shape[0]
        log(f"oracle water8k backward: senders {c1}/{N}, {done_b} edges, {t_b:.0f} s")
    return {"kind": "oracle", "dtype": "f64", "workload": "24,000-atom water box, whole", "part": part,
            "edges": E, "fwd_s": round(t_f, 1), "bwd_s": round(t_b, 1),
            "edges_per_s": round(E / (t_f + t_b), 1) if part == "both" else None,
            "chunk_nodes": chunk_nodes, "cpu": cpu_model(), "numpy": np.__version__,
            "torch_threads": torch.get_num_threads(), "affinity_cores": len(os.sched_getaffinity(0))}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-tp", action="store_true")
    ap.add_argument("--only", choices=["all", "conv", "generic", "radial", "bwd2", "linear", "tp", "ceiling",
                                       "capacity"],
                    default="all",
                    help="one section; 'capacity' (not part of 'all') times the 210,000-atom box at 64 channels, "
                         "which takes about 260 GB of device memory")
    ap.add_argument("--order", choices=["generated", "cell"], default="generated",
                    help="atom order of the water box: as generated (spatially random) or cell-sorted")
    ap.add_argument("--sweep", action="store_true",
                    help="also run the channel sweep at fixed node x channel count (the shape of the paper's "
                         "convolution throughput table); generates ten water boxes first")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the streaming probes that measure the HBM ceilings of the kernels' read:write mixes")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run one plain 2 GiB device copy (calibrates HBM byte counters)")
    ap.add_argument("--summarize-profiles", metavar="DIR",
                    help="only reduce the rocprofv3 CSV output under DIR to the profiles/ summaries, then exit")
    ap.add_argument("--oracle-water8k", choices=["both", "fwd", "bwd"],
                    help="only run the fp64 oracle once over the whole 24,000-atom water box (forward, backward or "
                         "both, in node chunks) on the host cores, print one JSON line, exit (both: about 15 "
                         "minutes on 16 cores)")
    ap.add_argument("--oracle-configs", action="store_true",
                    help="only time the fp64 oracle on the whole small workloads (64-atom cube, 1,000-molecule "
                         "water box, 200,000-row tensor product) on the host cores, print one JSON line, exit")
    args = ap.parse_args()
    if args.summarize_profiles:
        summarize_profiles(args.summarize_profiles)
        return
    if args.oracle_configs:
        print(json.dumps(oracle_configs()), flush=True)
        return
    if args.oracle_water8k:
        print(json.dumps(oracle_config4(args.oracle_water8k)), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              f"(the per-GPU kernel on its share is the unit measured)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_35099_amd import e3mi
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    e3mi.lib()
    dev = torch.device("cuda:0")
    out = {"metric": METRIC, "unit": "edges/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
           "data": "synthetic"}

    ceil = None
    if not args.no_ceiling and args.only in ("all", "ceiling"):
        ceil = hbm_ceilings(dev)
        out["ceiling"] = ceil
        if args.only == "ceiling":
            print(json.dumps(out), flush=True)
            return

    if args.only == "capacity":
        out["capacity"] = capacity(args, dev)
        print(json.dumps(out), flush=True)
        return

    # ---------------------------------------------------------------- conv
    cfg = synth.CONFIGS["water8k"]
    t0 = time.perf_counter()
    g = synth.graph(cfg, order=args.order)
    x = synth.node_features(cfg, g.n_nodes)
    dm = synth.out_cotangent(cfg, g.n_nodes)
    plan = e3mi.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    N, E, C = g.n_nodes, g.sender.shape[0], cfg.channels
    W = synth.bessel_matrix(cfg)
    s = torch.empty((E, plan.P, C), dtype=torch.float32, device=dev)
    for e0 in range(0, E, 1 << 16):
        e1 = min(E, e0 + (1 << 16))
        s[e0:e1].copy_(torch.from_numpy(synth.edge_weights(cfg, g.vec, e0, e1, W=W)))
    xs = torch.from_numpy(x).to(dev)
    dms = torch.from_numpy(dm).to(dev)
    vs = torch.from_numpy(g.vec).to(dev)
    snd = torch.from_numpy(g.sender).to(dev)
    rcv = torch.from_numpy(g.receiver).to(dev)
    log(f"inputs ready: N={N} E={E} ({time.perf_counter() - t0:.1f} s)")

    torch.cuda.synchronize()
    tg = []
    for _ in range(3):
        a = time.perf_counter()
        graph = e3mi.Graph(snd, rcv, N)
        torch.cuda.synchronize()
        tg.append((time.perf_counter() - a) * 1e3)
    m = torch.empty((N, plan.D_out, C), dtype=torch.float32, device=dev)
    dx = torch.empty((N, plan.D_in, C), dtype=torch.float32, device=dev)
    dvec = torch.empty((E, 3), dtype=torch.float32, device=dev)
    ds = torch.empty((E, plan.P, C), dtype=torch.float32, device=dev)
    ws = e3mi.workspace(e3mi.conv_workspace_size(plan, graph)[1])

    def step():
        e3mi.conv_fwd(plan, graph, xs, vs, s, out=m)
        e3mi.conv_bwd(plan, graph, xs, vs, s, dms, dx=dx, dvec=dvec, ds=ds, ws=ws)

    if args.only in ("all", "conv"):
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()
        e3mi.timing_reset()
        e3mi.timing_enable(True)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        torch.cuda.synchronize()
        ev0.record()
        for i in range(args.steps):
            marks[i].record()
            step()
        marks[-1].record()
        ev1.record()
        torch.cuda.synchronize()
        e3mi.timing_enable(False)
        per = e3mi.timing_read()
        ms_step = ev0.elapsed_time(ev1) / args.steps
        # per-step times: the paper's statistic (mean of the fastest 20%) and the median
        each = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
        fastest = each[:max(1, len(each) // 5)]
        kb, fwd_b, bwd_b = conv_bytes(N, E, C, plan.D_in, plan.D_out, plan.P)
        kernels = {}
        for name, (ms_tot, cnt) in per.items():
            ms_avg = ms_tot / cnt
            entry = {"ms": round(ms_avg, 4), "launches": cnt}
            if name in kb:
                entry["alg_GBps"] = round(kb[name] / (ms_avg * 1e-3) / 1e9, 1)
                entry["alg_bytes"] = kb[name]
            kernels[name] = entry
        dom = max((k for k in kernels if k in kb), key=lambda k: kernels[k]["ms"])
        ach = kb[dom] / (kernels[dom]["ms"] * 1e-3) / 1e9
        f_fwd, f_bwd = fma_counts(plan)
        kflops = {"conv_fwd": 2.0 * f_fwd * C * E, "conv_bwd_edges": 2.0 * f_bwd * C * E}
        for name in kflops:
            if name in kernels:
                tf = kflops[name] / (kernels[name]["ms"] * 1e-3) / 1e12
                kernels[name].update({"fma_per_edge_channel": f_fwd if name == "conv_fwd" else f_bwd,
                                      "TFLOPs": round(tf, 2), "valu_frac": round(tf / VALU_PEAK_TFLOPS, 4),
                                      "valu_busy_pct": counter_util(name, "VALUBusy")})
        if ceil:
            against_ceilings(kernels, ceil)
        dom_tf = kflops[dom] / (kernels[dom]["ms"] * 1e-3) / 1e12
        traffic = counter_traffic(dom)
        out.update({
            "value": E / (ms_step * 1e-3),
            "ms_per_step": ms_step,
            "config": {"workload": "water box, 8,000 rigid H2O = 24,000 atoms, periodic, r_c 5 A; "
                                   "x 128x0e+128x1o+128x2e+128x3o, harmonics l<=3, outputs l<=3, "
                                   "forward + backward convolution"
                                   + ("" if args.order == "generated" else "; atoms cell-sorted"),
                       "n_nodes": N, "n_edges": E, "channels": C, "paths": plan.P,
                       "D_in": plan.D_in, "D_out": plan.D_out},
            # the dominant sweep is bound by VALU issue (the kernels are compiled without packed fp32):
            # its FMA-equivalent work against the unpacked vector peak, with the HBM view beside it
            "roofline": {"bound": "alu", "kernel": dom, "achieved": round(dom_tf, 2), "peak": VALU_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(dom_tf / VALU_PEAK_TFLOPS, 4),
                         "traffic": traffic, "flops": kflops[dom],
                         "peak_packed_fp32": VALU_PEAK_PACKED_TFLOPS,
                         "frac_of_packed": round(dom_tf / VALU_PEAK_PACKED_TFLOPS, 4),
                         "valu_busy_pct": counter_util(dom, "VALUBusy"),
                         "hbm": {"achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                 "frac": round(ach / HBM_PEAK_GBS, 4), "alg_bytes": kb[dom],
                                 "counter_GBps": None if traffic is None else
                                 round(traffic / (kernels[dom]["ms"] * 1e-3) / 1e9, 1)}},
            "step_alg_GBps": round((fwd_b + bwd_b) / (ms_step * 1e-3) / 1e9, 1),
            # the step's kernels' committed counter bytes (HBM and fabric reads, all writes),
            # beside the algorithmic bytes: the difference is the dx partials' round trip and
            # the sender feature re-gathers
            "step_counter_bytes": step_counter_bytes(kernels),
            "step_counter_GBps": None if step_counter_bytes(kernels) is None else
            round(step_counter_bytes(kernels) / (ms_step * 1e-3) / 1e9, 1),
            "step_alg_frac": round((fwd_b + bwd_b) / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "fwd_alg_bytes": fwd_b, "bwd_alg_bytes": bwd_b,
            "kernels": kernels,
            "graph_build_ms": round(min(tg), 3),
            "step_ms_stats": {"median": round(each[len(each) // 2], 4),
                              "fastest_20pct_mean": round(sum(fastest) / len(fastest), 4),
                              "min": round(each[0], 4), "max": round(each[-1], 4)},
        })
        log(f"conv: {ms_step:.3f} ms/step, {E / ms_step / 1e3:.1f} M edges/s; kernels {kernels}")

    # ---------------------------------------------------------------- generic paths
    if args.only in ("all", "generic"):
        # the same step with the layout forced onto the two paths that serve
        # layouts without compiled kernels: generated single-block kinds run
        # block by block (composed), and the coupling records walked at run
        # time (records)
        for path in ("composed", "records"):
            gplan = e3mi.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out, records=path == "records",
                              composed=path == "composed")
            gws = e3mi.workspace(e3mi.conv_workspace_size(gplan, graph)[1])

            def gen_step():
                e3mi.conv_fwd(gplan, graph, xs, vs, s, out=m)
                e3mi.conv_bwd(gplan, graph, xs, vs, s, dms, dx=dx, dvec=dvec, ds=ds, ws=gws)

            for _ in range(args.warmup):
                gen_step()
            torch.cuda.synchronize()
            e3mi.timing_reset()
            e3mi.timing_enable(True)
            ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            nst = args.steps if path == "composed" else max(1, min(args.steps, 5))
            ev0.record()
            for _ in range(nst):
                gen_step()
            ev1.record()
            torch.cuda.synchronize()
            e3mi.timing_enable(False)
            per = e3mi.timing_read()
            g_ms = ev0.elapsed_time(ev1) / nst
            _, fwd_b, bwd_b = conv_bytes(N, E, C, plan.D_in, plan.D_out, plan.P)
            entry = {"ms_per_step": round(g_ms, 4), "edges_per_s": E / (g_ms * 1e-3), "steps": nst,
                     "step_alg_GBps": round((fwd_b + bwd_b) / (g_ms * 1e-3) / 1e9, 1),
                     "kernels": {k: {"ms_total_per_step": round(t / nst, 4), "launches": c}
                                 for k, (t, c) in per.items()}}
            if "ms_per_step" in out:
                entry["speed_vs_compiled"] = round(out["ms_per_step"] / g_ms, 4)
            out.setdefault("generic", {"workload": "the convolution step above with the layout forced onto the "
                                                   "paths for layouts without compiled kernels"})[path] = entry
            log(f"{path}: {g_ms:.3f} ms/step, {E / g_ms / 1e3:.1f} M edges/s; kernels {entry['kernels']}")
            del gws, gplan

    del ws, ds, s
    torch.cuda.empty_cache()

    # ---------------------------------------------------------------- fused radial weights
    if args.only in ("all", "radial"):
        h_np, W_np = synth.radial_inputs(cfg, g.vec)
        hs, Wd = torch.from_numpy(h_np).to(dev), torch.from_numpy(W_np).to(dev)
        K = W_np.shape[0]
        dh = torch.empty((E, K), dtype=torch.float32, device=dev)
        dW = torch.empty_like(Wd)
        rws = e3mi.workspace(e3mi.conv_radial_workspace_size(plan, graph, K))

        def rstep():
            e3mi.conv_fwd_radial(plan, graph, xs, vs, hs, Wd, out=m)
            e3mi.conv_bwd_radial(plan, graph, xs, vs, hs, Wd, dms, dx=dx, dvec=dvec, dh=dh, dW=dW, ws=rws)

        for _ in range(args.warmup):
            rstep()
        torch.cuda.synchronize()
        e3mi.timing_reset()
        e3mi.timing_enable(True)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record()
        for _ in range(args.steps):
            rstep()
        ev1.record()
        torch.cuda.synchronize()
        e3mi.timing_enable(False)
        per = e3mi.timing_read()
        r_ms = ev0.elapsed_time(ev1) / args.steps
        rf, rb = radial_bytes(N, E, C, plan.D_in, plan.D_out, plan.P, K)
        rk = {name: {"ms": round(t / c, 4), "launches": c} for name, (t, c) in per.items()}
        out["radial"] = {
            "workload": "as the convolution, with s = h W fused: h = 8-function Bessel basis of |r|, "
                        "W [8, P, C]", "K": K,
            "ms_per_step": round(r_ms, 4), "edges_per_s": E / (r_ms * 1e-3),
            "alg_bytes_fwd": rf, "alg_bytes_bwd": rb,
            "step_alg_GBps": round((rf + rb) / (r_ms * 1e-3) / 1e9, 1),
            "kernels": rk,
            # s = h W on the matrix cores, both sweeps: 2 K P C flops per edge each
            "radial_mfma_TFLOPs": round(2 * 2 * K * plan.P * C * E / (r_ms * 1e-3) / 1e12, 2),
        }
        log(f"radial: {r_ms:.3f} ms/step, {E / r_ms / 1e3:.1f} M edges/s; kernels {rk}")
        del rws, dh, dW, hs, Wd
    del dvec, dx, m
    torch.cuda.empty_cache()

    # ---------------------------------------------------------------- double backward
    if args.only in ("all", "bwd2"):
        ys = e3mi.sh(cfg.lmax_sh, vs)
        s2 = synth.normal_device(cfg.cid, 2, (E, plan.P, C), dev)
        dds = synth.normal_device(cfg.cid, 9, (E, plan.P, C), dev)
        ddx = synth.normal_device(cfg.cid, 10, (N, plan.D_in, C), dev)
        ddy = synth.normal_device(cfg.cid, 11, (E, plan.D_sh), dev)
        ws2 = e3mi.workspace(e3mi.conv_workspace_size(plan, graph)[1])
        for _ in range(args.warmup):
            outs = e3mi.conv_bwd2(plan, graph, xs, ys, s2, dms, ddx, ddy, dds, ws=ws2)
        del outs
        torch.cuda.synchronize()
        e3mi.timing_reset()
        e3mi.timing_enable(True)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record()
        for _ in range(args.steps):
            outs = e3mi.conv_bwd2(plan, graph, xs, ys, s2, dms, ddx, ddy, dds, ws=ws2)
        ev1.record()
        torch.cuda.synchronize()
        e3mi.timing_enable(False)
        per = e3mi.timing_read()
        b2_ms = ev0.elapsed_time(ev1) / args.steps
        f = 4
        nb = (N * (2 * plan.D_in + plan.D_out) * C * f + E * (2 * plan.D_sh + 2 * plan.P * C) * f   # inputs
              + N * (plan.D_in + plan.D_out) * C * f + E * (plan.D_sh + plan.P * C) * f)             # outputs
        out["bwd2"] = {"workload": "double backward of the convolution, same water box; ddx, ddy, dds N(0,1)",
                       "ms": round(b2_ms, 4), "edges_per_s": E / (b2_ms * 1e-3), "alg_bytes": nb,
                       "alg_GBps": round(nb / (b2_ms * 1e-3) / 1e9, 1),
                       "kernels": {k: {"ms_total_per_call": round(t / args.steps, 4), "launches": c}
                                   for k, (t, c) in per.items()}}
        log(f"bwd2: {b2_ms:.3f} ms, {out['bwd2']['alg_GBps']} GB/s; kernels {out['bwd2']['kernels']}")
        del outs, ws2
        # the same on the composed path (single-block kinds, fused sweeps per block)
        cplan = e3mi.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out, composed=True)
        wsc = e3mi.workspace(e3mi.conv_workspace_size(cplan, graph)[1])
        for _ in range(args.warmup):
            outs = e3mi.conv_bwd2(cplan, graph, xs, ys, s2, dms, ddx, ddy, dds, ws=wsc)
        del outs
        torch.cuda.synchronize()
        ev0.record()
        for _ in range(args.steps):
            outs = e3mi.conv_bwd2(cplan, graph, xs, ys, s2, dms, ddx, ddy, dds, ws=wsc)
        ev1.record()
        torch.cuda.synchronize()
        out["bwd2"]["composed_ms"] = round(ev0.elapsed_time(ev1) / args.steps, 4)
        log(f"bwd2 composed: {out['bwd2']['composed_ms']:.3f} ms")
        del outs, wsc, cplan, s2, dds, ddx, ddy, ys
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- linear mixing
    if args.only in ("all", "linear"):
        names = [f"{C}x{l3}{'e' if p3 > 0 else 'o'}" for (_, _, l3, p3, _, _, _) in plan.paths()]
        lin_in = "+".join(names)
        lin_out = "+".join(f"{C}x{l}{p}" for l in range(4) for p in "eo")
        L = e3mi.Linear(lin_in, lin_out)
        lx = synth.normal_device(4, 20, (N, L.D_in, L.C_in), dev)
        lW = synth.normal_device(4, 21, (L.n_weights,), dev) / 16
        ld = synth.normal_device(4, 22, (N, L.D_out, L.C_out), dev)
        ly = torch.empty((N, L.D_out, L.C_out), dtype=torch.float32, device=dev)
        ldx = torch.empty_like(lx)
        ldW = torch.empty_like(lW)
        lws = e3mi.workspace(L.workspace_size())
        for _ in range(args.warmup):
            L.forward(lx, lW, out=ly)
            L.backward(lx, lW, ld, dx=ldx, dW=ldW, ws=lws)
        torch.cuda.synchronize()
        e3mi.timing_reset()
        e3mi.timing_enable(True)
        for _ in range(args.steps):
            L.forward(lx, lW, out=ly)
            L.backward(lx, lW, ld, dx=ldx, dW=ldW, ws=lws)
        torch.cuda.synchronize()
        e3mi.timing_enable(False)
        per = e3mi.timing_read()
        # multiply-adds: every input row meets C_in x C_out weights (forward, dx and dW alike)
        flops = 2.0 * N * L.D_in * L.C_in * L.C_out
        lk = {}
        for name in ("linear_fwd", "linear_bwd_dx", "linear_bwd_dw", "linear_bwd_dw_sum"):
            if name in per:
                ms = per[name][0] / per[name][1]
                lk[name] = {"ms": round(ms, 4)}
                if name != "linear_bwd_dw_sum":
                    lk[name]["TFLOPs"] = round(flops / (ms * 1e-3) / 1e12, 2)
                    lk[name]["frac_fp32_mfma"] = round(flops / (ms * 1e-3) / 1e12 / 157.3, 4)
        out["linear"] = {"workload": f"equivariant mixing of the convolution output, {N} nodes: 34 path blocks "
                                     f"(D {L.D_in}) -> 8 irreps (D {L.D_out}), {C} -> {C} channels, fp32 MFMA",
                         "gflop_per_pass": round(flops / 1e9, 2),
                         "bound": "mfma", "peak_TFLOPs": 157.3, "kernels": lk}
        log(f"linear: {lk}")
        L.close()
        del lx, lW, ld, ly, ldx, ldW, lws
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- tp
    if not args.no_tp and args.only in ("all", "tp"):
        tcfg = synth.CONFIGS["tp200k"]
        tplan = e3mi.Plan(tcfg.irreps, tcfg.lmax_sh, tcfg.lmax_out)
        tx, tu, tw = synth.tp_inputs(tcfg)
        txd, twd = torch.from_numpy(tx).to(dev), torch.from_numpy(tw).to(dev)
        ty = e3mi.sh(tcfg.lmax_sh, torch.from_numpy(tu).to(dev))
        R = tx.shape[0]
        tz = torch.empty((R, tplan.D_out, tplan.C), dtype=torch.float32, device=dev)
        for _ in range(args.warmup):
            e3mi.tp_fwd(tplan, txd, ty, twd, out=tz)
        torch.cuda.synchronize()
        e3mi.timing_reset()
        e3mi.timing_enable(True)
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record()
        for _ in range(args.steps):
            e3mi.tp_fwd(tplan, txd, ty, twd, out=tz)
        a1.record()
        torch.cuda.synchronize()
        e3mi.timing_enable(False)
        tk = e3mi.timing_read()["tp_fwd"]
        t_ms = tk[0] / tk[1]
        nb = tp_bytes(R, tplan.C, tplan.D_in, tplan.D_sh, tplan.D_out, tplan.P)
        out["tp"] = {"workload": "200,000 rows, x 128x0e+128x1o+128x2e, harmonics l<=3, outputs l<=3",
                     "ms": round(t_ms, 4), "rows_per_s": R / (t_ms * 1e-3),
                     "alg_GBps": round(nb / (t_ms * 1e-3) / 1e9, 1),
                     "frac": round(nb / (t_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4), "alg_bytes": nb,
                     "event_ms": round(a0.elapsed_time(a1) / args.steps, 4)}
        if ceil:
            kk = {"tp_fwd": {"ms": t_ms}}
            against_ceilings(kk, ceil)
            out["tp"].update({k: v for k, v in kk["tp_fwd"].items() if k != "ms"})
        log(f"tp: {t_ms:.3f} ms, {out['tp']['alg_GBps']} GB/s")
        del tz
        tdz = synth.normal_device(tcfg.cid, synth._DM, (R, tplan.D_out, tplan.C), dev)
        tdx, tdw = torch.empty_like(txd), torch.empty_like(twd)
        tdy = torch.empty_like(ty)
        tws = e3mi.workspace(e3mi.tp_workspace_size(tplan, R))
        for _ in range(args.warmup):
            e3mi.tp_bwd(tplan, txd, ty, twd, tdz, tdx, tdy, tdw, tws)
        torch.cuda.synchronize()
        e3mi.timing_reset()
        e3mi.timing_enable(True)
        a0.record()
        for _ in range(args.steps):
            e3mi.tp_bwd(tplan, txd, ty, twd, tdz, tdx, tdy, tdw, tws)
        a1.record()
        torch.cuda.synchronize()
        e3mi.timing_enable(False)
        tt = e3mi.timing_read()
        tb_ms = tt["tp_bwd"][0] / tt["tp_bwd"][1]
        nb = tp_bwd_bytes(R, tplan.C, tplan.D_in, tplan.D_sh, tplan.D_out, tplan.P)
        out["tp_bwd"] = {"workload": out["tp"]["workload"], "ms": round(tb_ms, 4),
                         "dy_sum_ms": round(tt["tp_bwd_dy"][0] / tt["tp_bwd_dy"][1], 4),
                         "rows_per_s": R / (tb_ms * 1e-3),
                         "alg_GBps": round(nb / (tb_ms * 1e-3) / 1e9, 1),
                         "frac": round(nb / (tb_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4), "alg_bytes": nb,
                         "event_ms": round(a0.elapsed_time(a1) / args.steps, 4)}
        if ceil:
            kk = {"tp_bwd": {"ms": tb_ms}}
            against_ceilings(kk, ceil)
            out["tp_bwd"].update({k: v for k, v in kk["tp_bwd"].items() if k != "ms"})
        log(f"tp_bwd: {tb_ms:.3f} ms, {out['tp_bwd']['alg_GBps']} GB/s")
        # the same product through the caller-supplied record path (the plan's records, unweighted)
        i0, i1, i2, rv = tplan.records()
        rtp = e3mi.RecordTP(tplan.D_in, tplan.D_sh, tplan.D_out, i0, i1, i2, rv, False)
        tz = torch.empty((R, tplan.D_out, tplan.C), dtype=torch.float32, device=dev)
        for _ in range(args.warmup):
            rtp.forward(txd, ty, out=tz)
        torch.cuda.synchronize()
        e3mi.timing_reset()
        e3mi.timing_enable(True)
        for _ in range(args.steps):
            rtp.forward(txd, ty, out=tz)
        torch.cuda.synchronize()
        e3mi.timing_enable(False)
        tt = e3mi.timing_read()
        tg_ms = tt["tpg_fwd"][0] / tt["tpg_fwd"][1]
        nb = R * (tplan.D_in * tplan.C + tplan.D_sh + tplan.D_out * tplan.C) * 4
        out["tp_records"] = {"workload": out["tp"]["workload"] + ", unweighted, records streamed at run time",
                             "nnz": int(i0.shape[0]), "ms": round(tg_ms, 4),
                             "alg_GBps": round(nb / (tg_ms * 1e-3) / 1e9, 1)}
        log(f"tp_records: {tg_ms:.3f} ms, {out['tp_records']['alg_GBps']} GB/s")
        rtp.close()
        del tz
        del tdz, tdx, tdw, tdy, tws, txd, twd, ty

    if args.sweep:
        out["sweep"] = sweep(args, dev)

    if args.copy_probe:
        n = (2 << 30) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        dst.copy_(src)
        c1.record()
        torch.cuda.synchronize()
        out["copy_probe"] = {"bytes_each_way": 2 << 30, "ms": round(c0.elapsed_time(c1), 4),
                             "GBps_rw": round(2 * (2 << 30) / (c0.elapsed_time(c1) * 1e-3) / 1e9, 1)}
        del src, dst

    # ---------------------------------------------------------------- cpu
    if not args.no_cpu_baseline and args.only in ("all", "conv"):
        out["cpu_baseline"] = cpu_baseline(cfg, g, x, dm)
        log(f"cpu baseline: {out['cpu_baseline']['value']:.1f} edges/s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
