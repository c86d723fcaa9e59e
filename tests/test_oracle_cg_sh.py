"""Pins of the oracle's coupling coefficients and harmonics against facts that
do not come from the oracle itself: sympy's exact Clebsch-Gordan values,
scipy's complex harmonics, textbook closed forms, group-theoretic identities.
"""
import os
from math import sqrt

import numpy as np
import pytest
from sympy import S
from sympy.physics.wigner import clebsch_gordan

from oracle import cg, sh, wigner

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "closed_forms.txt")


def _golden(kind):
    out = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        parts = line.split(None, 3 if kind == "sh" else 4)
        if parts[0] == kind:
            out.append(parts[1:])
    return out


def _unit(rng, n):
    g = rng.standard_normal((n, 3))
    return g / np.linalg.norm(g, axis=1, keepdims=True)


# ---------------------------------------------------------------- complex CG
def test_racah_equals_sympy():
    worst = 0.0
    for l1 in range(4):
        for l2 in range(4):
            for L in range(abs(l1 - l2), l1 + l2 + 1):
                for m1 in range(-l1, l1 + 1):
                    for m2 in range(-l2, l2 + 1):
                        M = m1 + m2
                        if abs(M) > L:
                            continue
                        ref = float(clebsch_gordan(S(l1), S(l2), S(L), S(m1), S(m2), S(M)))
                        worst = max(worst, abs(cg.cg_complex(l1, m1, l2, m2, L, M) - ref))
    assert worst < 1e-14


def test_complex_cg_unitary_and_special_values():
    for l1 in range(4):
        for l2 in range(4):
            rows = []
            for L in range(abs(l1 - l2), l1 + l2 + 1):
                rows.append(cg.cg_complex_block(l1, l2, L).reshape(2 * L + 1, -1))
            U = np.concatenate(rows, axis=0)
            n = (2 * l1 + 1) * (2 * l2 + 1)
            assert U.shape == (n, n)
            assert np.abs(U @ U.T - np.eye(n)).max() < 1e-14
            # stretched state
            assert abs(cg.cg_complex(l1, l1, l2, l2, l1 + l2, l1 + l2) - 1.0) < 1e-15
    for l in range(4):
        for m in range(-l, l + 1):
            ref = (-1) ** (l - m) / sqrt(2 * l + 1)
            assert abs(cg.cg_complex(l, m, l, -m, 0, 0) - ref) < 1e-15


# ---------------------------------------------------------------- harmonics
def test_sh_golden_closed_forms():
    rng = np.random.default_rng(0)
    u = _unit(rng, 64)
    Y = sh.sh_unit(2, u)
    x, y, z = u[:, 0], u[:, 1], u[:, 2]
    env = {"sqrt": np.sqrt, "x": x, "y": y, "z": z}
    n = 0
    for l, m, expr in _golden("sh"):
        l, m = int(l), int(m)
        ref = eval(expr, {"__builtins__": {}}, env) * np.ones_like(x)
        assert np.abs(Y[:, l * l + l + m] - ref).max() < 1e-14, (l, m)
        n += 1
    assert n == 9


def test_sh_against_scipy_complex():
    """Textbook real-from-complex relation, with scipy's harmonics (CS phase):
    m>0: sqrt2 (-1)^m Re Y^m, m<0: sqrt2 (-1)^m Im Y^|m|, m=0: Y^0; then the
    y-polar axes of the adopted convention."""
    rng = np.random.default_rng(1)
    u = _unit(rng, 200)
    # evaluate the textbook real functions at the permuted point v = (u_z, u_x, u_y)
    v = np.stack([u[:, 2], u[:, 0], u[:, 1]], axis=1)
    Y = sh.sh_unit(3, u)
    for l in range(4):
        Yc = cg.sh_complex_unit(l, v)
        for m in range(-l, l + 1):
            if m > 0:
                ref = sqrt(2) * (-1) ** m * Yc[:, l + m].real
            elif m < 0:
                ref = sqrt(2) * (-1) ** m * Yc[:, l - m].imag
            else:
                ref = Yc[:, l].real
            assert np.abs(Y[:, l * l + l + m] - ref).max() < 1e-12, (l, m)


def test_sh_identities():
    rng = np.random.default_rng(2)
    u = _unit(rng, 500)
    Y = sh.sh_unit(3, u)
    for l in range(4):
        blk = Y[:, l * l:(l + 1) ** 2]
        assert np.abs((blk ** 2).sum(1) - (2 * l + 1)).max() < 1e-12      # addition theorem
        par = sh.sh_unit(3, -u)[:, l * l:(l + 1) ** 2]
        assert np.abs(par - (-1) ** l * blk).max() < 1e-13              # parity
    # Monte-Carlo orthogonality on a large sample (component normalisation: E[Y Y^T] = I)
    u = _unit(np.random.default_rng(3), 400_000)
    Y = sh.sh_unit(3, u)
    G = Y.T @ Y / u.shape[0]
    assert np.abs(G - np.eye(16)).max() < 0.03


def test_sh_harmonic_polynomials():
    """|r|^l Y_l(r/|r|) is a harmonic polynomial (Laplacian zero), App. A.2."""
    import torch
    rng = np.random.default_rng(4)
    r = torch.tensor(rng.standard_normal((20, 3)), requires_grad=True)
    P = sh.sh_poly(3, r)
    for i in range(16):
        g, = torch.autograd.grad(P[:, i].sum(), r, create_graph=True)
        lap = 0
        for d in range(3):
            h, = torch.autograd.grad(g[:, d].sum(), r, retain_graph=True)
            lap = lap + h[:, d]
        assert lap.abs().max().item() < 1e-10, i


def test_sh_vjp_finite_difference():
    rng = np.random.default_rng(5)
    vec = rng.standard_normal((10, 3)) * 2.0
    dy = rng.standard_normal((10, 16))
    g = sh.sh_vec_vjp(3, vec, dy)
    h = 1e-6
    for d in range(3):
        e = np.zeros(3)
        e[d] = h
        fd = ((sh.sh_vec(3, vec + e) - sh.sh_vec(3, vec - e)) * dy).sum(1) / (2 * h)
        assert np.abs(fd - g[:, d]).max() < 1e-7
    # degree-0 homogeneity: the gradient is orthogonal to the edge vector
    assert np.abs((g * vec).sum(1)).max() < 1e-12


# ---------------------------------------------------------------- Wigner-D
def test_wigner_group_law():
    rng = np.random.default_rng(6)
    R1, R2 = wigner.random_rotation(rng), wigner.random_rotation(rng)
    for l in range(4):
        D1, D2 = wigner.wigner_d(l, R1), wigner.wigner_d(l, R2)
        D12 = wigner.wigner_d(l, R1 @ R2)
        assert np.abs(D1 @ D1.T - np.eye(2 * l + 1)).max() < 1e-12
        assert abs(np.linalg.det(D1) - 1.0) < 1e-12
        assert np.abs(D12 - D1 @ D2).max() < 1e-12
    assert np.abs(wigner.wigner_d(1, R1) - R1).max() < 1e-12   # Y_1 = sqrt3 u


# ---------------------------------------------------------------- real CG
def _all_paths():
    for l1 in range(4):
        for l2 in range(4):
            for l3 in range(abs(l1 - l2), min(l1 + l2, 3) + 1):
                yield l1, l2, l3


def test_real_cg_orthonormal_and_equivariant():
    rng = np.random.default_rng(7)
    R = wigner.random_rotation(rng)
    D = [wigner.wigner_d(l, R) for l in range(4)]
    for l1, l2, l3 in _all_paths():
        C = cg.cg_real_block(l1, l2, l3)
        Cm = C.reshape(2 * l3 + 1, -1)
        assert np.abs(Cm @ Cm.T - np.eye(2 * l3 + 1)).max() < 1e-13
        lhs = np.einsum("Mab,ai,bj->Mij", C, D[l1], D[l2])
        rhs = np.einsum("MN,Nij->Mij", D[l3], C)
        assert np.abs(lhs - rhs).max() < 1e-12, (l1, l2, l3)


def test_real_cg_golden_closed_forms():
    eps = np.zeros((3, 3, 3))
    for a, b, c in [(0, 1, 2), (1, 2, 0), (2, 0, 1)]:
        eps[a, b, c], eps[a, c, b] = 1.0, -1.0
    forms = {"dot_over_sqrt3": lambda: np.eye(3)[None] / sqrt(3),
             "cross_over_sqrt2": lambda: eps / sqrt(2)}
    n = 0
    for l1, l2, l3, name in _golden("cg"):
        l1, l2, l3 = int(l1), int(l2), int(l3)
        C = cg.cg_real_block(l1, l2, l3)
        if name == "identity":
            if l1 == 0:
                ref = np.eye(2 * l3 + 1)[:, None, :]
            else:
                ref = np.eye(2 * l3 + 1)[:, :, None]
        else:
            ref = forms[name]()
        assert np.abs(C - ref).max() < 1e-14, (l1, l2, l3)
        n += 1
    assert n == 8


def test_real_cg_couples_harmonics_of_one_vector():
    """sum C[M,a,b] Y_l1(u)_a Y_l2(u)_b = +-sqrt((2l1+1)(2l2+1)/(2l3+1)) <l1 0 l2 0|l3 0> Y_l3(u)_M.

    (Product of two harmonics of the same direction, projected on degree l3;
    zero when l1+l2+l3 is odd.)  Ties the coupling tables to the harmonics.
    """
    rng = np.random.default_rng(8)
    u = _unit(rng, 50)
    Y = sh.sh_unit(6, u)
    for l1, l2, l3 in _all_paths():
        C = cg.cg_real_block(l1, l2, l3)
        lhs = np.einsum("Mab,na,nb->nM", C, Y[:, l1 * l1:(l1 + 1) ** 2], Y[:, l2 * l2:(l2 + 1) ** 2])
        kappa = sqrt((2 * l1 + 1) * (2 * l2 + 1) / (2 * l3 + 1)) * cg.cg_complex(l1, 0, l2, 0, l3, 0)
        ref = Y[:, l3 * l3:(l3 + 1) ** 2]
        if (l1 + l2 + l3) % 2:
            assert np.abs(lhs).max() < 1e-12
        else:
            ok = min(np.abs(lhs - kappa * ref).max(), np.abs(lhs + kappa * ref).max())
            assert ok < 1e-12, (l1, l2, l3)
