"""Real spherical harmonics of edge vectors, and their vector-Jacobian product.

Part of the test-only fp64 oracle; see the package docstring.

Follows App. A.2 ("Harmonic polynomials": the degree-l harmonics are the
harmonic homogeneous polynomials of degree l, a basis of the irrep Y_l) and
App. A.3 ("Harmonics": an edge vector is expanded as the concatenation of the
banks Y_l, l = 0..lmax, each bank m = -l..l).

The paper fixes neither normalisation nor axes.  Reading adopted here:

  * S_l^m is the textbook real solid harmonic in Cartesian form (no
    Condon-Shortley sign in the real functions): for m > 0 it is proportional
    to Re (x+iy)^m, for m < 0 to Im (x+iy)^|m|, times the polynomial
        Pi_l^m(z, r) = sqrt((l-m)!/(l+m)!) *
            sum_k (-1)^k 2^-l C(l,k) C(2l-2k,l) (l-2k)!/(l-2k-m)! r^2k z^(l-2k-m)
    with prefactor sqrt(2l+1) * (sqrt 2 if m != 0), so that on the unit
    sphere sum_m S_l^m(u)^2 = 2l+1 ("component" normalisation);
  * the harmonics used by the method are Y_l(u) = S_l(u_z, u_x, u_y), i.e.
    the y axis is the polar axis.  Then Y_0 = 1 and Y_1(u) = sqrt(3) u.

The Jacobian of r -> Y(r/|r|) is taken by float64 autograd of the same
formula (a library primitive); no derivative is written by hand.
"""
from __future__ import annotations

from math import comb, factorial, sqrt

import numpy as np
import torch


def _pi_coeffs(l: int, m: int):
    """Coefficients of Pi_l^m as a list of (k, coefficient) pairs."""
    pre = sqrt(factorial(l - m) / factorial(l + m))
    out = []
    for k in range((l - m) // 2 + 1):
        c = ((-1) ** k) * (2.0 ** -l) * comb(l, k) * comb(2 * l - 2 * k, l) \
            * factorial(l - 2 * k) / factorial(l - 2 * k - m)
        out.append((k, pre * c))
    return out


def solid_real(l: int, x: torch.Tensor, y: torch.Tensor, z: torch.Tensor) -> torch.Tensor:
    """Homogeneous real solid harmonics S_l^m(x,y,z), m = -l..l, last axis.

    Evaluated on the unit sphere this is the component-normalised real
    spherical harmonic in the textbook axes (z polar).
    """
    r2 = x * x + y * y + z * z
    # A_m + i B_m = (x + i y)^m by the recurrence of complex multiplication.
    A = [torch.ones_like(x)]
    B = [torch.zeros_like(x)]
    for _ in range(l):
        a, b = A[-1], B[-1]
        A.append(x * a - y * b)
        B.append(x * b + y * a)
    cols = []
    for m in range(-l, l + 1):
        am = abs(m)
        pi = torch.zeros_like(x)
        for k, c in _pi_coeffs(l, am):
            pi = pi + c * r2 ** k * z ** (l - 2 * k - am)
        norm = sqrt(2 * l + 1) * (sqrt(2.0) if m != 0 else 1.0)
        if m > 0:
            cols.append(norm * pi * A[am])
        elif m < 0:
            cols.append(norm * pi * B[am])
        else:
            cols.append(norm * pi)
    return torch.stack(cols, dim=-1)


def _as_t(a):
    if isinstance(a, torch.Tensor):
        return a.to(torch.float64), False
    return torch.as_tensor(np.asarray(a, dtype=np.float64)), True


def sh_unit(lmax: int, u):
    """Y(u) = concat_l Y_l(u) for unit vectors u [..., 3] -> [..., (lmax+1)^2]."""
    ut, was_np = _as_t(u)
    ux, uy, uz = ut[..., 0], ut[..., 1], ut[..., 2]
    out = torch.cat([solid_real(l, uz, ux, uy) for l in range(lmax + 1)], dim=-1)
    return out.numpy() if was_np else out


def sh_poly(lmax: int, r):
    """The homogeneous polynomials |r|^l Y_l(r/|r|) (used for harmonicity checks)."""
    return sh_unit(lmax, r)  # the formula is homogeneous in (x, y, z)


def sh_vec(lmax: int, vec):
    """Y(vec/|vec|) for edge vectors vec [..., 3] (float64)."""
    vt, was_np = _as_t(vec)
    n = torch.linalg.vector_norm(vt, dim=-1, keepdim=True)
    out = sh_unit(lmax, vt / n)
    return out.numpy() if was_np else out


def sh_vec_vjp(lmax: int, vec, dy):
    """dvec = (dY/dvec)^T dy for Y(vec/|vec|), by float64 autograd."""
    vt, was_np = _as_t(vec)
    dyt, _ = _as_t(dy)
    vt = vt.detach().clone().requires_grad_(True)
    with torch.enable_grad():
        n = torch.linalg.vector_norm(vt, dim=-1, keepdim=True)
        y = sh_unit(lmax, vt / n)
        (g,) = torch.autograd.grad(y, vt, grad_outputs=dyt)
    g = g.detach()
    return g.numpy() if was_np else g
