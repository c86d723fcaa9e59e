"""Clebsch-Gordan coefficients: complex (Racah) and real (in the harmonics' basis).

Part of the test-only fp64 oracle; see the package docstring.

Follows App. A.3 ("Tensor product": (x (x) y)^{LM} = sum_{m+m'=M}
C^{LM}_{lm,l'm'} x^{lm} y^{l'm'}) and App. G.2, which builds the same
coefficients by ladder operators.  The oracle deliberately does NOT use the
ladder construction: it uses Racah's closed formula, an independent route.

Readings adopted where the paper is silent (the GPU-side builder applies the
same conventions by its own code):

  1. Normalisation: the complex coefficients are the standard unitary
     (Condon-Shortley) ones; no extra path normalisation factor.
  2. Real basis: the real coupling tensor of a path (l1, l2, l3) is
        C_real[M, a, b] = sum U3[M, M'] C[M'; m1, m2] conj(U1[a, m1]) conj(U2[b, m2])
     where U_l is the change of basis real = U_l . complex, fitted by least
     squares on sample points (the fit is exact).  The complex harmonics are
     scipy's (Condon-Shortley phase), times sqrt(4 pi).
  3. Each real block is real or purely imaginary; an imaginary block is
     multiplied by -i.  Canonical sign: the first entry with |c| > 1e-12 in
     row-major (M, a, b) order is made positive.
"""
from __future__ import annotations

from fractions import Fraction
from functools import lru_cache
from math import factorial, pi, sqrt

import numpy as np
from scipy.special import sph_harm_y

from . import sh as _sh


def cg_complex(l1: int, m1: int, l2: int, m2: int, L: int, M: int) -> float:
    """<l1 m1 l2 m2 | L M> by Racah's formula (exact rationals, one sqrt)."""
    if M != m1 + m2:
        return 0.0
    if not (abs(l1 - l2) <= L <= l1 + l2):
        return 0.0
    if abs(m1) > l1 or abs(m2) > l2 or abs(M) > L:
        return 0.0
    f = factorial
    pre = Fraction((2 * L + 1) * f(L + l1 - l2) * f(L - l1 + l2) * f(l1 + l2 - L),
                   f(l1 + l2 + L + 1))
    pre *= f(L + M) * f(L - M) * f(l1 - m1) * f(l1 + m1) * f(l2 - m2) * f(l2 + m2)
    s = Fraction(0)
    for k in range(0, l1 + l2 - L + 1):
        args = (k, l1 + l2 - L - k, l1 - m1 - k, l2 + m2 - k, L - l2 + m1 + k, L - l1 - m2 + k)
        if min(args) < 0:
            continue
        den = 1
        for a in args:
            den *= f(a)
        s += Fraction((-1) ** k, den)
    if s == 0:
        return 0.0
    val = sqrt(float(pre * s * s))
    return val if s > 0 else -val


@lru_cache(maxsize=None)
def cg_complex_block(l1: int, l2: int, L: int) -> np.ndarray:
    """C[M, m1, m2] for M = -L..L, m1 = -l1..l1, m2 = -l2..l2."""
    out = np.zeros((2 * L + 1, 2 * l1 + 1, 2 * l2 + 1))
    for M in range(-L, L + 1):
        for m1 in range(-l1, l1 + 1):
            m2 = M - m1
            if abs(m2) <= l2:
                out[M + L, m1 + l1, m2 + l2] = cg_complex(l1, m1, l2, m2, L, M)
    return out


def sh_complex_unit(l: int, u: np.ndarray) -> np.ndarray:
    """Complex harmonics Y_l^m(u), m = -l..l, Condon-Shortley, times sqrt(4 pi)."""
    u = np.asarray(u, dtype=np.float64)
    theta = np.arccos(np.clip(u[..., 2], -1.0, 1.0))
    phi = np.arctan2(u[..., 1], u[..., 0])
    cols = [sph_harm_y(l, m, theta, phi) for m in range(-l, l + 1)]
    return np.sqrt(4 * pi) * np.stack(cols, axis=-1)


@lru_cache(maxsize=None)
def real_basis(l: int) -> np.ndarray:
    """U_l with Y_l(u) = U_l @ Ycomplex_l(u), fitted by least squares."""
    rng = np.random.default_rng(1000 + l)
    g = rng.standard_normal((8 * (2 * l + 1) + 16, 3))
    u = g / np.linalg.norm(g, axis=1, keepdims=True)
    yr = _sh.sh_unit(l, u)[:, l * l:]          # [K, 2l+1] real, our axes
    yc = sh_complex_unit(l, u)                 # [K, 2l+1] complex
    # yr = yc @ U^T  ->  least squares for U^T
    ut, res, rank, _ = np.linalg.lstsq(yc, yr.astype(np.complex128), rcond=None)
    U = ut.T
    resid = np.abs(yc @ ut - yr).max()
    if rank != 2 * l + 1 or resid > 1e-10:
        raise AssertionError(f"real-basis fit failed for l={l}: rank {rank} resid {resid}")
    return U


def canonical_sign(block: np.ndarray) -> np.ndarray:
    """Make the first |entry| > 1e-12 in row-major order positive."""
    flat = block.reshape(-1)
    for v in flat:
        if abs(v) > 1e-12:
            return block if v > 0 else -block
    return block


@lru_cache(maxsize=None)
def cg_real_block(l1: int, l2: int, l3: int) -> np.ndarray:
    """Real coupling tensor C[M, a, b] of path (l1, l2, l3) in the harmonics' basis."""
    C = cg_complex_block(l1, l2, l3).astype(np.complex128)
    U1, U2, U3 = real_basis(l1), real_basis(l2), real_basis(l3)
    R = np.einsum("MN,Nij,ai,bj->Mab", U3, C, U1.conj(), U2.conj())
    re, im = np.abs(R.real).max(), np.abs(R.imag).max()
    if im > re:
        R = -1j * R
    if np.abs(R.imag).max() > 1e-13:
        raise AssertionError(f"coupling ({l1},{l2},{l3}) is not real up to a phase")
    out = np.ascontiguousarray(R.real)
    out[np.abs(out) < 1e-13] = 0.0   # exact zeros of the coupling, not rounding noise
    return canonical_sign(out)


def path_blocks(lay) -> list[np.ndarray]:
    """Real coupling tensor for every path of a layout (oracle.irreps.Layout)."""
    return [cg_real_block(p.l1, p.l2, p.l3) for p in lay.paths]


def coo_records(lay, tol: float = 1e-12):
    """Unfolded sparse records (i0, i1, i2, value) of App. E.2, sorted by i0.

    i0 runs over D_out, i1 over D_in, i2 over D_sh.  Used to compare with the
    GPU-side builder's table and to count non-zeros.
    """
    recs = []
    for p, blk in zip(lay.paths, path_blocks(lay)):
        for M in range(blk.shape[0]):
            for a in range(blk.shape[1]):
                for b in range(blk.shape[2]):
                    v = blk[M, a, b]
                    if abs(v) > tol:
                        recs.append((p.out_off + M, p.x_off + a, p.y_off + b, float(v)))
    recs.sort(key=lambda r: (r[0], r[1], r[2]))
    return recs


def dense_tensor(lay) -> np.ndarray:
    """The full dense coupling tensor [D_out, D_in, D_sh] (tiny layouts only)."""
    T = np.zeros((lay.d_out, lay.d_in, lay.d_sh))
    for i0, i1, i2, v in coo_records(lay, tol=0.0):
        T[i0, i1, i2] = v
    return T
