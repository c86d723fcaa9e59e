"""The generated per-edge contraction code, compiled for the host and checked
against the fp64 oracle on the CPU.

The table generator's output (the straight-line code that the GPU sweeps run
per edge and channel: pre-contraction A = C . y, the forward contraction with
the path weight, and the backward's cotangents of x, s and y through every
contraction order the generator picks) is plain C++ apart from a few device
qualifiers.  Here it is built with g++ next to a small driver that runs the
forward and backward groups of one edge and one channel, and the results are
compared with the oracle's weighted tensor product and its backward
(App. E.1, eq. tp-bwd) on random inputs, for every compiled variant and every
single-block kind of the composed path (and the double backward's three-term
sweeps of both)."""
import ctypes as ct
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import irreps as oirreps
from oracle import sh as osh
from oracle import tp as otp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_35099_amd", "csrc")

# tag of the generated variant -> (x blocks, lmax_sh, lmax_out, parity)
VARIANTS = {
    "V_x01_s2_o2": ("0e+1o", 2, 2, "all"),
    "V_x012_s2_o2": ("0e+1o+2e", 2, 2, "all"),
    "V_x01_s3_o3": ("0e+1o", 3, 3, "all"),
    "V_x012_s3_o3": ("0e+1o+2e", 3, 3, "all"),
    "V_x0123_s3_o3": ("0e+1o+2e+3o", 3, 3, "all"),
    "V_x0e1o_s2_o2_n": ("0e+1o", 2, 2, "natural"),
    "V_x0e1o_s3_o3_n": ("0e+1o", 3, 3, "natural"),
    "V_x0e1o2e_s3_o3_n": ("0e+1o+2e", 3, 3, "natural"),
    "V_x0e1o2e3o_s3_o3_n": ("0e+1o+2e+3o", 3, 3, "natural"),
    "V_x1032_s3_o3": ("1o+0e+3o+2e", 3, 3, "all"),
}


def _kind_layout(tag):
    """The single-block layout a kind tag names: K_l<l1>_s<lsh>_o<lout>_<a|n|p>
    (all paths; natural-parity paths of a block of parity (-1)^l1; of the
    other parity)."""
    _, l, sh, o, cls = tag.split("_")
    l1, lsh, lout = int(l[1:]), int(sh[1:]), int(o[1:])
    even = (l1 % 2 == 0) == (cls != "p")
    irreps = f"1x{l1}{'e' if even else 'o'}"
    return oirreps.layout(irreps, lsh, lout, parity="all" if cls == "a" else "natural"), lsh


def _kind_tags():
    """The kinds the generator should emit: every single x block of degree
    <= 3 (all paths, or the natural-parity ones of either block parity) under
    harmonics and outputs to degree 3, one per distinct (path list, harmonics
    degree), in the generator's enumeration order."""
    seen, tags = set(), []
    for l1 in range(4):
        for lsh in range(4):
            for lout in range(4):
                for cls in "anp":
                    tag = f"K_l{l1}_s{lsh}_o{lout}_{cls}"
                    lay, _ = _kind_layout(tag)
                    key = (tuple((p.l1, p.l2, p.l3) for p in lay.paths), lsh)
                    if lay.n_paths and key not in seen:
                        seen.add(key)
                        tags.append(tag)
    return tags


KINDS = _kind_tags()


def _layout(tag):
    if tag.startswith("K_"):
        return _kind_layout(tag)
    blocks, lsh, lout, parity = VARIANTS[tag]
    irreps = "+".join("1x" + b for b in blocks.split("+"))
    return oirreps.layout(irreps, lsh, lout, parity=parity), lsh

DRIVER = r"""
#include <cmath>
#define __device__
#define __forceinline__ inline
#define __restrict__
struct alignas(16) float4 { float x, y, z, w; };
struct alignas(32) double4 { double x, y, z, w; };
#define E3_FWD_PIN() ((void)0)
#define __builtin_amdgcn_sched_barrier(x) ((void)0)
#include "variants.inc"
using namespace e3gen;

template <class V, int G>
void fwd_groups(const float* Y, const float* x, const float* s, float* m) {
  if constexpr (G < V::NFG) {
    using F = typename V::template FG<G>;
    alignas(16) float A[F::NA];
    F::make_A(Y, A);
    float xv[F::NXR][1], sv[F::NPATH][1], acc[F::NROW][1];
    for (int i = 0; i < F::NXR; ++i) xv[i][0] = x[F::XROW[i]];
    for (int i = 0; i < F::NPATH; ++i) sv[i][0] = s[F::PATH[i]];
    for (int i = 0; i < F::NROW; ++i) acc[i][0] = 0.0f;
    F::template edge<1>(A, xv, sv, acc);
    for (int i = 0; i < F::NROW; ++i) m[F::OROW[i]] = acc[i][0];
    fwd_groups<V, G + 1>(Y, x, s, m);
  }
}

template <class V, int G>
void fwd3_groups(const float* Y, const float* Yd, const float* x, const float* xd, const float* s, const float* sd,
                 float* m) {
  if constexpr (G < V::NFG) {
    using F = typename V::template FG<G>;
    alignas(16) float A[F::NA], A2[F::NA];
    F::make_A(Y, A);
    F::make_A(Yd, A2);
    float xv[F::NXR][1], xdv[F::NXR][1], sv[F::NPATH][1], sdv[F::NPATH][1], acc[F::NROW][1];
    for (int i = 0; i < F::NXR; ++i) xv[i][0] = x[F::XROW[i]], xdv[i][0] = xd[F::XROW[i]];
    for (int i = 0; i < F::NPATH; ++i) sv[i][0] = s[F::PATH[i]], sdv[i][0] = sd[F::PATH[i]];
    for (int i = 0; i < F::NROW; ++i) acc[i][0] = 0.0f;
    F::template edge3<1>(A, A2, xv, xdv, sv, sdv, acc);
    for (int i = 0; i < F::NROW; ++i) m[F::OROW[i]] = acc[i][0];
    fwd3_groups<V, G + 1>(Y, Yd, x, xd, s, sd, m);
  }
}

template <class V, int G>
void bwd_groups(const float* Y, const float* x, const float* s, const float* dm, float* dx, float* dy,
                float* ds) {
  if constexpr (G < V::NBG) {
    using B = typename V::template BG<G>;
    alignas(16) float A[B::NA];
    B::make_A(Y, A);
    float Yv[V::D_SH], dyl[V::D_SH];
    for (int i = 0; i < V::D_SH; ++i) Yv[i] = Y[i], dyl[i] = 0.0f;
    float xv[B::NXR][1], sv[B::NPATH][1], dmv[B::NROW][1], t[B::NXR][1];
    for (int i = 0; i < B::NXR; ++i) xv[i][0] = x[B::XROW[i]], t[i][0] = 0.0f;
    for (int i = 0; i < B::NPATH; ++i) sv[i][0] = s[B::PATH[i]];
    for (int i = 0; i < B::NROW; ++i) dmv[i][0] = dm[B::OROW[i]];
    auto st = [&](int pl, const float (&v)[1]) { ds[B::PATH[pl]] = v[0]; };
    B::template edge<false, 1>(A, Yv, xv, sv, dmv, t, dyl, st);
    for (int i = 0; i < B::NXR; ++i) dx[B::XROW[i]] += t[i][0];
    for (int i = 0; i < V::D_SH; ++i) dy[i] += dyl[i];
    bwd_groups<V, G + 1>(Y, x, s, dm, dx, dy, ds);
  }
}

template <class V, int G>
void bwd3_groups(const float* Y, const float* Y2, const float* x, const float* xd, const float* s, const float* sd,
                 const float* dm, float* gx, float* gy, float* gs) {
  if constexpr (G < V::NBG) {
    using B = typename V::template BG<G>;
    float Yv[V::D_SH], Y2v[V::D_SH], dyl[V::D_SH];
    for (int i = 0; i < V::D_SH; ++i) Yv[i] = Y[i], Y2v[i] = Y2[i], dyl[i] = 0.0f;
    float xv[B::NXR][1], xdv[B::NXR][1], sv[B::NPATH][1], sdv[B::NPATH][1], dmv[B::NROW][1], t[B::NXR][1];
    for (int i = 0; i < B::NXR; ++i) xv[i][0] = x[B::XROW[i]], xdv[i][0] = xd[B::XROW[i]], t[i][0] = 0.0f;
    for (int i = 0; i < B::NPATH; ++i) sv[i][0] = s[B::PATH[i]], sdv[i][0] = sd[B::PATH[i]];
    for (int i = 0; i < B::NROW; ++i) dmv[i][0] = dm[B::OROW[i]];
    auto st = [&](int pl, const float (&v)[1]) { gs[B::PATH[pl]] = v[0]; };
    B::template edge3<1>(Yv, Y2v, xv, xdv, sv, sdv, dmv, t, dyl, st);
    for (int i = 0; i < B::NXR; ++i) gx[B::XROW[i]] += t[i][0];
    for (int i = 0; i < V::D_SH; ++i) gy[i] += dyl[i];
    bwd3_groups<V, G + 1>(Y, Y2, x, xd, s, sd, dm, gx, gy, gs);
  }
}

#define E3_HOST_ENTRY(V)                                                                        \
  extern "C" void V##_fwd(const float* Y, const float* x, const float* s, float* m) {          \
    fwd_groups<V, 0>(Y, x, s, m);                                                              \
  }                                                                                            \
  extern "C" void V##_fwd3(const float* Y, const float* Yd, const float* x, const float* xd, const float* s, \
                           const float* sd, float* m) {                                        \
    fwd3_groups<V, 0>(Y, Yd, x, xd, s, sd, m);                                                 \
  }                                                                                            \
  extern "C" void V##_bwd3(const float* Y, const float* Y2, const float* x, const float* xd,    \
                           const float* s, const float* sd, const float* dm, float* gx, float* gy,  \
                           float* gs) {                                                        \
    for (int i = 0; i < V::D_IN; ++i) gx[i] = 0.0f;                                            \
    for (int i = 0; i < V::D_SH; ++i) gy[i] = 0.0f;                                            \
    bwd3_groups<V, 0>(Y, Y2, x, xd, s, sd, dm, gx, gy, gs);                                    \
  }                                                                                            \
  extern "C" void V##_bwd(const float* Y, const float* x, const float* s, const float* dm,      \
                          float* dx, float* dy, float* ds) {                                   \
    for (int i = 0; i < V::D_IN; ++i) dx[i] = 0.0f;                                            \
    for (int i = 0; i < V::D_SH; ++i) dy[i] = 0.0f;                                            \
    bwd_groups<V, 0>(Y, x, s, dm, dx, dy, ds);                                                 \
  }
E3GEN_FOR_EACH_VARIANT(E3_HOST_ENTRY)

// single-block kinds (their strides are the composed path's business; the
// per-edge code is the same)
#include "kinds.inc"
E3GEN_FOR_EACH_KIND(E3_HOST_ENTRY)
extern "C" const char* e3_kind_list() {
  return ""
#define E3_KIND_NAME(V) #V " "
  E3GEN_FOR_EACH_KIND(E3_KIND_NAME);
}
"""


@pytest.fixture(scope="module")
def hostlib(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("needs g++")
    d = tmp_path_factory.mktemp("genhost")
    exe = str(d / "e3gen")
    subprocess.run(["g++", "-O1", "-std=c++17", "-o", exe, os.path.join(CSRC, "gen.cpp"),
                    os.path.join(CSRC, "builder.cpp")], check=True)
    subprocess.run([exe, str(d)], check=True)
    (d / "driver.cpp").write_text(DRIVER)
    so = str(d / "libgenhost.so")
    subprocess.run(["g++", "-O1", "-std=c++17", "-ffp-contract=off", "-shared", "-fPIC", "-I", str(d), "-o", so,
                    str(d / "driver.cpp")], check=True)
    return ct.CDLL(so)


def _ptr(a):
    return a.ctypes.data_as(ct.c_void_p)


def _rel(a, b):
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(np.asarray(a, dtype=np.float64) - b) / max(np.linalg.norm(b), 1e-300))


@pytest.mark.parametrize("tag", sorted(VARIANTS))
def test_generated_edge_code_matches_oracle(hostlib, tag):
    lay, lsh = _layout(tag)
    rng = np.random.default_rng(11)
    R = 24
    u = rng.standard_normal((R, 3))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    y = np.asarray(osh.sh_unit(lsh, u), dtype=np.float32)
    x = rng.standard_normal((R, lay.d_in)).astype(np.float32)
    s = rng.standard_normal((R, lay.n_paths)).astype(np.float32)
    dm = rng.standard_normal((R, lay.d_out)).astype(np.float32)
    fwd, bwd = getattr(hostlib, f"{tag}_fwd"), getattr(hostlib, f"{tag}_bwd")
    m = np.zeros((R, lay.d_out), np.float32)
    dx = np.zeros((R, lay.d_in), np.float32)
    dy = np.zeros((R, lay.d_sh), np.float32)
    ds = np.zeros((R, lay.n_paths), np.float32)
    for r in range(R):
        rows = [np.ascontiguousarray(a[r]) for a in (y, x, s, dm)]
        outs = [np.zeros_like(a[r]) for a in (m, dx, dy, ds)]
        fwd(_ptr(rows[0]), _ptr(rows[1]), _ptr(rows[2]), _ptr(outs[0]))
        bwd(_ptr(rows[0]), _ptr(rows[1]), _ptr(rows[2]), _ptr(rows[3]), _ptr(outs[1]), _ptr(outs[2]),
            _ptr(outs[3]))
        m[r], dx[r], dy[r], ds[r] = outs
    # one channel per row: the oracle's channel axis has length 1
    ref_m = otp.tp(lay, x[:, :, None], y, s[:, :, None]).numpy()[:, :, 0]
    ref_dx, ref_dy, ref_dw = otp.tp_bwd(lay, x[:, :, None], y, s[:, :, None], dm[:, :, None])
    assert _rel(m, ref_m) < 1e-6
    assert _rel(dx, ref_dx.numpy()[:, :, 0]) < 1e-6
    assert _rel(ds, ref_dw.numpy()[:, :, 0]) < 1e-6
    assert _rel(dy, ref_dy.numpy()) < 1e-6


@pytest.mark.parametrize("tag", sorted(VARIANTS) + KINDS)
def test_generated_three_term_forward_matches_oracle(hostlib, tag):
    """The double backward's output cotangent in one pass: the sum of three
    forward products, with the x, harmonic and weight tangents in turn."""
    lay, lsh = _layout(tag)
    rng = np.random.default_rng(12)
    R = 16
    u = rng.standard_normal((R, 3))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    y = np.asarray(osh.sh_unit(lsh, u), dtype=np.float32)
    yd = rng.standard_normal((R, lay.d_sh)).astype(np.float32)
    x, xd = (rng.standard_normal((R, lay.d_in)).astype(np.float32) for _ in range(2))
    s, sd = (rng.standard_normal((R, lay.n_paths)).astype(np.float32) for _ in range(2))
    fwd3 = getattr(hostlib, f"{tag}_fwd3")
    m = np.zeros((R, lay.d_out), np.float32)
    for r in range(R):
        rows = [np.ascontiguousarray(a[r]) for a in (y, yd, x, xd, s, sd)]
        out = np.zeros(lay.d_out, np.float32)
        fwd3(*[_ptr(a) for a in rows], _ptr(out))
        m[r] = out
    c = lambda a: a[:, :, None]
    ref = (otp.tp(lay, c(xd), y, c(s)) + otp.tp(lay, c(x), yd, c(s)) + otp.tp(lay, c(x), y, c(sd))).numpy()[:, :, 0]
    assert _rel(m, ref) < 1e-6


@pytest.mark.parametrize("tag", sorted(VARIANTS) + KINDS)
def test_generated_three_term_backward_matches_oracle(hostlib, tag):
    """The double backward's three backward products in one pass: ds of
    (xd, y, s) and of (x, y2, s), dy of (xd, y, s) and of (x, y, sd), and the
    x cotangents of (x, y2, s) and of (x, y, sd)."""
    lay, lsh = _layout(tag)
    rng = np.random.default_rng(13)
    R = 16
    u = rng.standard_normal((R, 3))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    y = np.asarray(osh.sh_unit(lsh, u), dtype=np.float32)
    y2 = rng.standard_normal((R, lay.d_sh)).astype(np.float32)
    x, xd = (rng.standard_normal((R, lay.d_in)).astype(np.float32) for _ in range(2))
    s, sd = (rng.standard_normal((R, lay.n_paths)).astype(np.float32) for _ in range(2))
    dm = rng.standard_normal((R, lay.d_out)).astype(np.float32)
    bwd3 = getattr(hostlib, f"{tag}_bwd3")
    gx = np.zeros((R, lay.d_in), np.float32)
    gy = np.zeros((R, lay.d_sh), np.float32)
    gs = np.zeros((R, lay.n_paths), np.float32)
    for r in range(R):
        rows = [np.ascontiguousarray(a[r]) for a in (y, y2, x, xd, s, sd, dm)]
        outs = [np.zeros_like(a[r]) for a in (gx, gy, gs)]
        bwd3(*[_ptr(a) for a in rows], *[_ptr(a) for a in outs])
        gx[r], gy[r], gs[r] = outs
    c = lambda a: a[:, :, None]
    dx_a, dy_a, dw_a = otp.tp_bwd(lay, c(xd), y, c(s), c(dm))   # (xd, y, s)
    dx_b, dy_b, dw_b = otp.tp_bwd(lay, c(x), y2, c(s), c(dm))   # (x, y2, s)
    dx_c, dy_c, dw_c = otp.tp_bwd(lay, c(x), y, c(sd), c(dm))   # (x, y, sd)
    assert _rel(gs, (dw_a + dw_b).numpy()[:, :, 0]) < 1e-6
    assert _rel(gy, (dy_a + dy_c).numpy()) < 1e-6
    assert _rel(gx, (dx_b + dx_c).numpy()[:, :, 0]) < 1e-6


def test_generated_kind_code_matches_oracle(hostlib):
    """Every single-block kind the composed path runs: its per-edge forward and
    backward code against the oracle's tensor product of that block alone, and
    the set of kinds covers every block of degree <= 3 under harmonics and
    outputs to degree 3 (each block's path list has a kind)."""
    hostlib.e3_kind_list.restype = ct.c_char_p
    tags = hostlib.e3_kind_list().decode().split()
    assert tags == KINDS
    have = set()
    for tag in tags:
        lay, lsh = _kind_layout(tag)
        assert lay.n_paths > 0, tag
        have.add((tuple((p.l1, p.l2, p.l3) for p in lay.paths), lsh))
        rng = np.random.default_rng(17)
        R = 6
        u = rng.standard_normal((R, 3))
        u /= np.linalg.norm(u, axis=1, keepdims=True)
        y = np.asarray(osh.sh_unit(lsh, u), dtype=np.float32)
        x = rng.standard_normal((R, lay.d_in)).astype(np.float32)
        s = rng.standard_normal((R, lay.n_paths)).astype(np.float32)
        dm = rng.standard_normal((R, lay.d_out)).astype(np.float32)
        fwd, bwd = getattr(hostlib, f"{tag}_fwd"), getattr(hostlib, f"{tag}_bwd")
        m = np.zeros((R, lay.d_out), np.float32)
        dx = np.zeros((R, lay.d_in), np.float32)
        dy = np.zeros((R, lay.d_sh), np.float32)
        ds = np.zeros((R, lay.n_paths), np.float32)
        for r in range(R):
            rows = [np.ascontiguousarray(a[r]) for a in (y, x, s, dm)]
            outs = [np.zeros_like(a[r]) for a in (m, dx, dy, ds)]
            fwd(_ptr(rows[0]), _ptr(rows[1]), _ptr(rows[2]), _ptr(outs[0]))
            bwd(_ptr(rows[0]), _ptr(rows[1]), _ptr(rows[2]), _ptr(rows[3]), _ptr(outs[1]), _ptr(outs[2]),
                _ptr(outs[3]))
            m[r], dx[r], dy[r], ds[r] = outs
        ref_m = otp.tp(lay, x[:, :, None], y, s[:, :, None]).numpy()[:, :, 0]
        ref_dx, ref_dy, ref_dw = otp.tp_bwd(lay, x[:, :, None], y, s[:, :, None], dm[:, :, None])
        assert _rel(m, ref_m) < 1e-6, tag
        assert _rel(dx, ref_dx.numpy()[:, :, 0]) < 1e-6, tag
        assert _rel(ds, ref_dw.numpy()[:, :, 0]) < 1e-6, tag
        assert _rel(dy, ref_dy.numpy()) < 1e-6, tag
    # coverage: every block (degree, parity) of degree <= 3, each parity rule,
    # harmonics and outputs to degree 3
    for l1 in range(4):
        for p in "eo":
            for lsh in range(4):
                for lout in range(4):
                    for parity in ("all", "natural"):
                        lay = oirreps.layout(f"1x{l1}{p}", lsh, lout, parity=parity)
                        if lay.n_paths:
                            key = (tuple((q.l1, q.l2, q.l3) for q in lay.paths), lsh)
                            assert key in have, (l1, p, lsh, lout, parity)
