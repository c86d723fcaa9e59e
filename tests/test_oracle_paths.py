"""Pins of the oracle's path enumeration and real coupling tables.

The path lists and counts in tests/golden/paths.txt were written by hand from
App. A.3's triangle rule, App. B.1's parity product and the enumeration order
(no code produced them).  The real coupling tensors are rebuilt here by a route
that shares nothing with the oracle's: sympy's complex Clebsch-Gordan
coefficients turned real with the textbook change of basis (z as the polar
axis), instead of Racah's formula with a basis fitted on sample points of the
oracle's own harmonics (y as the polar axis).  The two bases differ by a
proper rotation applied to every degree alike, so each path's tensor must be
the same up to its overall sign.

Dropping the pseudo-parity paths, an off-by-one in the l3 range, a different
block order or a lost coefficient each fail one of these tests.
"""
import os
from functools import lru_cache

import numpy as np
import pytest

from oracle import cg as ocg
from oracle import irreps as oirreps

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paths.txt")


def _golden():
    cases, paths = {}, {}
    for line in open(GOLDEN):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        tok = line.split()
        if tok[0] == "case":
            name, irreps, lsh, lout, parity = tok[1], tok[2], int(tok[3]), int(tok[4]), tok[5]
            kv = dict(t.split("=") for t in tok[6:])
            cases[name] = (irreps, lsh, lout, parity, {k: int(v) for k, v in kv.items()})
            paths[name] = []
        elif tok[0] == "path":
            l1p = tok[2]
            paths[tok[1]].append((int(l1p[:-1]), 1 if l1p[-1] == "e" else -1, int(tok[3]), int(tok[4])))
        else:
            raise ValueError(line)
    return cases, paths


CASES, PATHS = _golden()


def _textbook_U(l):
    """Real harmonics from the complex (Condon-Shortley) ones, textbook form."""
    U = np.zeros((2 * l + 1, 2 * l + 1), complex)
    r2 = 1 / np.sqrt(2)
    for m in range(-l, l + 1):
        if m > 0:
            U[m + l, -m + l] += r2
            U[m + l, m + l] += r2 * (-1) ** m
        elif m == 0:
            U[l, l] = 1
        else:
            a = -m
            U[m + l, -a + l] += 1j * r2
            U[m + l, a + l] += -1j * r2 * (-1) ** a
    return U


@lru_cache(maxsize=None)
def _textbook_block(l1, l2, l3):
    from sympy.physics.wigner import clebsch_gordan
    C = np.zeros((2 * l3 + 1, 2 * l1 + 1, 2 * l2 + 1))
    for M in range(-l3, l3 + 1):
        for m1 in range(-l1, l1 + 1):
            m2 = M - m1
            if abs(m2) <= l2:
                C[M + l3, m1 + l1, m2 + l2] = float(clebsch_gordan(l1, l2, l3, m1, m2, M))
    R = np.einsum("MN,Nij,ai,bj->Mab", _textbook_U(l3), C, _textbook_U(l1).conj(), _textbook_U(l2).conj())
    if np.abs(R.imag).max() > np.abs(R.real).max():
        R = -1j * R
    assert np.abs(R.imag).max() < 1e-12
    return R.real


def _independent_counts(lay):
    nnz, pairs = 0, set()
    for p in lay.paths:
        blk = _textbook_block(p.l1, p.l2, p.l3)
        for M, a, b in zip(*np.nonzero(np.abs(blk) > 1e-12)):
            nnz += 1
            pairs.add((p.out_off + M, p.x_off + a))
    return nnz, len(pairs)


@pytest.mark.parametrize("name", sorted(CASES))
def test_layout_matches_hand_enumeration(name):
    irreps, lsh, lout, parity, want = CASES[name]
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    assert lay.n_paths == want["P"]
    assert lay.d_out == want["D_out"]
    got = [(p.l1, p.p1, p.l2, p.l3) for p in lay.paths]
    if PATHS[name]:
        assert got == PATHS[name]
    out = 0
    for k, p in enumerate(lay.paths):
        assert p.k == k and p.out_off == out and p.y_off == p.l2 * p.l2
        assert p.p3 == p.p1 * (-1) ** p.l2          # App. B.1
        assert abs(p.l1 - p.l2) <= p.l3 <= min(p.l1 + p.l2, lout)   # App. A.3
        if parity == "natural":
            assert p.p3 == (-1) ** p.l3
        out += 2 * p.l3 + 1


@pytest.mark.parametrize("name", sorted(CASES))
def test_record_counts(name):
    irreps, lsh, lout, parity, want = CASES[name]
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    recs = ocg.coo_records(lay)
    nnz, npairs = len(recs), len({(r[0], r[1]) for r in recs})
    assert (nnz, npairs) == _independent_counts(lay)
    if "nnz" in want:
        assert nnz == want["nnz"] and npairs == want["pairs"]


def test_real_coupling_equals_textbook_basis_up_to_sign():
    for l1 in range(4):
        for l2 in range(4):
            for l3 in range(abs(l1 - l2), min(l1 + l2, 3) + 1):
                a = _textbook_block(l1, l2, l3)
                b = ocg.cg_real_block(l1, l2, l3)
                i = int(np.argmax(np.abs(a)))
                sign = np.sign(a.flat[i]) * np.sign(b.flat[i])
                assert np.abs(sign * a - b).max() < 1e-12, (l1, l2, l3)


def test_pseudo_parity_paths_are_kept_by_default():
    # 1o x 1o -> 1e is triangle-allowed with p3 = +1 != (-1)^1: kept under "all",
    # dropped under "natural"
    lay = oirreps.layout("1x1o", 1, 1)
    assert [(p.l2, p.l3, p.p3) for p in lay.paths] == [(0, 1, -1), (1, 0, 1), (1, 1, 1)]
    nat = oirreps.layout("1x1o", 1, 1, parity="natural")
    assert [(p.l2, p.l3) for p in nat.paths] == [(0, 1), (1, 0)]
