"""Seeded synthetic inputs for the channelwise CG convolution and tensor product.

This package is the ONE module shared by the HIP path's tests/benchmark and by
the fp64 oracle.  It holds geometry, random numbers and array shapes only:
none of the method's arithmetic (no harmonics, no coupling coefficients, no
contraction).  The per-edge weights of the water boxes are built from a random
radial basis (a Bessel basis of the edge length times a fixed random matrix),
which is input synthesis, not part of the operation under test.

Every random stream is ``numpy.random.default_rng(SeedSequence([seed, stream,
chunk]))`` so that any chunk of any array can be regenerated on its own (the
oracle checks large workloads on sampled rows).  Values are drawn in float64
and rounded to float32, the precision both sides consume.

Workloads (shapes of those the method is benchmarked on), by name:

  cube64    tiny conv: 64 atoms uniform in a non-periodic cube at 0.1 atoms/A^3,
            all ordered pairs closer than 4 A; x 8x0e+8x1o, harmonics l<=2,
            output l<=2; x, s, dm ~ N(0,1).  Edges in sender-major order.
  tp200k    standalone tensor product: 200,000 rows of x 128x0e+128x1o+128x2e,
            random unit vectors (harmonics l<=3), per-row path weights ~ N(0,1).
  water1k   water box, 1,000 rigid H2O at 1 g/cm^3, periodic, r_c = 5 A; x
            128x0e+128x1o; s = Bessel_8(|r|) @ W.  Edges in receiver-major order.
  water8k   same construction, 8,000 H2O (24,000 atoms); x 128x0e+...+128x3o.
  water70k  70,000 H2O (210,000 atoms), 64 channels, s ~ N(0,1).
"""
from __future__ import annotations

from dataclasses import dataclass
from math import pi

import numpy as np

# streams
_GEOM, _X, _S, _DM, _W, _VEC = 0, 1, 2, 3, 4, 5

MOLECULES_PER_A3 = 0.033428   # liquid water at 1 g/cm^3
R_OH = 0.9572
ANGLE_HOH = 104.52 * pi / 180.0
R_CUT = 5.0
MIN_INTERMOLECULAR = 1.0
N_BESSEL = 8


@dataclass(frozen=True)
class Config:
    cid: int
    kind: str          # "conv" or "tp"
    irreps: str
    lmax_sh: int
    lmax_out: int
    channels: int
    n_mol: int = 0     # water boxes
    n_atoms: int = 0   # uniform cube of atoms
    rows: int = 0      # tensor product rows
    weights: str = "normal"   # "normal" or "bessel"
    edge_order: str = "receiver"
    r_cut: float = R_CUT


def sweep_config(lmax: int, channels: int) -> Config:
    """Channel sweep at a fixed product of node count and channel count (2^21 at
    l_max 3, 2^22 at l_max 2) on water boxes with ~45 neighbours per atom
    (r_c = 4.75 A at liquid density): x = C x (0e+1o+...+l_max), harmonics and
    outputs up to l_max, N(0,1) edge weights."""
    n_atoms = (1 << (21 if lmax == 3 else 22)) // channels
    irreps = "+".join(f"{channels}x{l}{'e' if l % 2 == 0 else 'o'}" for l in range(lmax + 1))
    return Config(100 + 10 * lmax + channels.bit_length(), "conv", irreps, lmax, lmax, channels,
                  n_mol=n_atoms // 3, r_cut=4.75)


# Workloads by name (the number is the seed of each one's random streams).
CONFIGS = {
    "cube64": Config(1, "conv", "8x0e+8x1o", 2, 2, 8, n_atoms=64, edge_order="sender"),
    "tp200k": Config(2, "tp", "128x0e+128x1o+128x2e", 3, 3, 128, rows=200_000),
    "water1k": Config(3, "conv", "128x0e+128x1o", 3, 3, 128, n_mol=1000, weights="bessel"),
    "water8k": Config(4, "conv", "128x0e+128x1o+128x2e+128x3o", 3, 3, 128, n_mol=8000,
              weights="bessel"),
    "water70k": Config(5, "conv", "64x0e+64x1o+64x2e+64x3o", 3, 3, 64, n_mol=70_000),
}


def rng(cid: int, stream: int, chunk: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([cid, stream, chunk]))


def irreps_dims(irreps: str):
    """(D_in, channels) of an irreps string; shape bookkeeping only."""
    dim, muls = 0, set()
    for tok in irreps.split("+"):
        mul, rest = tok.split("x")
        muls.add(int(mul))
        dim += 2 * int(rest[:-1]) + 1
    assert len(muls) == 1
    return dim, muls.pop()


def n_paths_dout(irreps: str, lmax_sh: int, lmax_out: int):
    """Number of paths and output rows (shape bookkeeping for array sizes)."""
    P = D = 0
    for tok in irreps.split("+"):
        l1 = int(tok.split("x")[1][:-1])
        for l2 in range(lmax_sh + 1):
            for l3 in range(abs(l1 - l2), min(l1 + l2, lmax_out) + 1):
                P += 1
                D += 2 * l3 + 1
    return P, D


# --------------------------------------------------------------------------
# geometry
# --------------------------------------------------------------------------

def _random_rotations(g: np.random.Generator, n: int) -> np.ndarray:
    q = g.standard_normal((n, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    w, x, y, z = q.T
    R = np.empty((n, 3, 3))
    R[:, 0, 0] = 1 - 2 * (y * y + z * z)
    R[:, 0, 1] = 2 * (x * y - z * w)
    R[:, 0, 2] = 2 * (x * z + y * w)
    R[:, 1, 0] = 2 * (x * y + z * w)
    R[:, 1, 1] = 1 - 2 * (x * x + z * z)
    R[:, 1, 2] = 2 * (y * z - x * w)
    R[:, 2, 0] = 2 * (x * z - y * w)
    R[:, 2, 1] = 2 * (y * z + x * w)
    R[:, 2, 2] = 1 - 2 * (x * x + y * y)
    return R


def _molecule_atoms(O: np.ndarray, R: np.ndarray) -> np.ndarray:
    h = 0.5 * ANGLE_HOH
    body = np.array([[0.0, 0.0, 0.0],
                     [R_OH * np.sin(h), 0.0, R_OH * np.cos(h)],
                     [-R_OH * np.sin(h), 0.0, R_OH * np.cos(h)]])
    return O[:, None, :] + np.einsum("nij,aj->nai", R, body)


def _pairs_within(pos: np.ndarray, L: float | None, rc: float, cell: float | None = None):
    """All unordered pairs (i<j) closer than rc; minimum image if L is given.

    Returns (i, j, d) with d = pos[j] - pos[i] (minimum image).
    """
    n = pos.shape[0]
    cw = rc if cell is None else max(cell, rc)
    if L is None:
        lo = pos.min(axis=0)
        span = pos.max(axis=0) - lo + 1e-9
        nc = np.maximum((span // cw).astype(int), 1)
        cellw = span / nc
        cell3 = np.minimum(((pos - lo) / cellw).astype(int), nc - 1)
    else:
        nc = np.array([max(int(L // cw), 1)] * 3)
        cellw = L / nc
        cell3 = np.minimum((np.mod(pos, L) / cellw).astype(int), nc - 1)
    ncell = int(np.prod(nc))
    cid = (cell3[:, 0] * nc[1] + cell3[:, 1]) * nc[2] + cell3[:, 2]
    order = np.argsort(cid, kind="stable")
    counts = np.bincount(cid, minlength=ncell)
    start = np.concatenate([[0], np.cumsum(counts)])
    occ = int(counts.max())
    table = np.full((ncell, occ), -1, dtype=np.int64)
    slot = np.arange(n) - start[cid[order]]
    table[cid[order], slot] = order
    offs = [(a, b, c) for a in (-1, 0, 1) for b in (-1, 0, 1) for c in (-1, 0, 1)]
    c3 = np.stack(np.unravel_index(np.arange(ncell), tuple(nc)), axis=1)
    I, J, D = [], [], []
    seen = set()
    small = bool(np.any(nc < 3))
    for off in offs:
        nb3 = c3 + np.array(off)
        if L is None:
            ok = np.all((nb3 >= 0) & (nb3 < nc), axis=1)
        else:
            ok = np.ones(ncell, dtype=bool)
            nb3 = np.mod(nb3, nc)
        nb = np.ravel_multi_index(tuple(nb3[ok].T), tuple(nc)) if ok.any() else np.zeros(0, int)
        src = np.nonzero(ok)[0]
        if small:
            # avoid visiting the same (cell, neighbour-cell) pair twice when nc < 3
            keys = src * ncell + nb
            fresh = np.array([k not in seen for k in keys.tolist()], dtype=bool)
            seen.update(keys[fresh].tolist())
            src, nb = src[fresh], nb[fresh]
        step = max(256, (1 << 21) // (occ * occ))
        for c0 in range(0, src.shape[0], step):
            a = table[src[c0:c0 + step]]
            b = table[nb[c0:c0 + step]]
            ia = np.broadcast_to(a[:, :, None], (a.shape[0], occ, occ))
            ib = np.broadcast_to(b[:, None, :], (a.shape[0], occ, occ))
            valid = (ia >= 0) & (ib >= 0) & (ia < ib)
            ia, ib = ia[valid], ib[valid]
            d = pos[ib] - pos[ia]
            if L is not None:
                d -= L * np.round(d / L)
            r = np.linalg.norm(d, axis=1)
            close = r < rc
            I.append(ia[close])
            J.append(ib[close])
            D.append(d[close])
    if not I:
        return np.zeros(0, int), np.zeros(0, int), np.zeros((0, 3))
    I, J, D = np.concatenate(I), np.concatenate(J), np.concatenate(D)
    if not small:
        return I, J, D
    # a pair can be found through two different cell offsets when nc < 3
    key = I * n + J
    _, first = np.unique(key, return_index=True)
    return I[first], J[first], D[first]


def water_box(cid: int, n_mol: int):
    """Rigid waters, uniform positions and orientations, periodic cube.

    Rejection: no two atoms of different molecules closer than 1.0 A.
    Returns (positions [3*n_mol, 3], L).
    """
    g = rng(cid, _GEOM)
    L = (n_mol / MOLECULES_PER_A3) ** (1.0 / 3.0)
    O = g.uniform(0.0, L, size=(n_mol, 3))
    R = _random_rotations(g, n_mol)
    for _ in range(1000):
        atoms = _molecule_atoms(O, R).reshape(-1, 3)
        i, j, _d = _pairs_within(atoms, L, MIN_INTERMOLECULAR, cell=2.5)
        bad = (i // 3) != (j // 3)
        if not bad.any():
            return np.mod(atoms, L), L
        redo = np.unique(np.maximum(i[bad] // 3, j[bad] // 3))
        O[redo] = g.uniform(0.0, L, size=(redo.shape[0], 3))
        R[redo] = _random_rotations(g, redo.shape[0])
    raise RuntimeError("water box rejection did not converge")


def uniform_cube(cid: int, n_atoms: int, density: float = 0.1):
    g = rng(cid, _GEOM)
    L = (n_atoms / density) ** (1.0 / 3.0)
    return g.uniform(0.0, L, size=(n_atoms, 3)), L


@dataclass
class Graph:
    n_nodes: int
    sender: np.ndarray    # int32 [E]
    receiver: np.ndarray  # int32 [E]
    vec: np.ndarray       # float32 [E, 3], pos[receiver] - pos[sender] (+ image shift)
    box: float | None


def cell_order(pos: np.ndarray, L: float, n_mol: int, cell: float = R_CUT) -> np.ndarray:
    """Atom permutation that sorts whole molecules by the cell of their oxygen
    (cells of side ~r_c, visited in Morton order), keeping O, H, H together."""
    nc = max(int(L // cell), 1)
    c3 = np.minimum((np.mod(pos[0::3], L) / (L / nc)).astype(np.int64), nc - 1)
    code = np.zeros(n_mol, dtype=np.int64)
    for bit in range(12):
        for a in range(3):
            code |= ((c3[:, a] >> bit) & 1) << (3 * bit + a)
    mol = np.argsort(code, kind="stable")
    return (3 * mol[:, None] + np.arange(3)[None, :]).reshape(-1)


def graph(cfg: Config, order: str = "generated") -> Graph:
    """Edge list of a workload.  order="cell" renumbers the atoms of a water
    box so that molecules are sorted by spatial cell (the as-generated order is
    spatially random)."""
    if cfg.n_atoms:
        pos, L = uniform_cube(cfg.cid, cfg.n_atoms)
        i, j, d = _pairs_within(pos, None, 4.0)
        box = None
        n = cfg.n_atoms
    else:
        pos, L = water_box(cfg.cid, cfg.n_mol)
        if order == "cell":
            pos = pos[cell_order(pos, L, cfg.n_mol)]
        i, j, d = _pairs_within(pos, L, cfg.r_cut)
        box = L
        n = pos.shape[0]
    # both directions: edge (i -> j) carries pos[j]-pos[i]; (j -> i) the negative
    snd = np.concatenate([i, j])
    rcv = np.concatenate([j, i])
    vec = np.concatenate([d, -d])
    if cfg.edge_order == "sender":
        order = np.lexsort((rcv, snd))
    else:
        order = np.lexsort((snd, rcv))
    return Graph(n, snd[order].astype(np.int32), rcv[order].astype(np.int32),
                 vec[order].astype(np.float32), box)


# --------------------------------------------------------------------------
# features
# --------------------------------------------------------------------------

def normal_f32(cid: int, stream: int, shape, chunk: int = 0) -> np.ndarray:
    return rng(cid, stream, chunk).standard_normal(shape).astype(np.float32)


def node_features(cfg: Config, n_nodes: int) -> np.ndarray:
    d_in, C = irreps_dims(cfg.irreps)
    return normal_f32(cfg.cid, _X, (n_nodes, d_in, C))


def out_cotangent(cfg: Config, n_nodes: int) -> np.ndarray:
    _, d_out = n_paths_dout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    return normal_f32(cfg.cid, _DM, (n_nodes, d_out, cfg.channels))


def bessel_matrix(cfg: Config) -> np.ndarray:
    P, _ = n_paths_dout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    return rng(cfg.cid, _W).standard_normal((N_BESSEL, P * cfg.channels)) / np.sqrt(N_BESSEL)


def bessel_basis(r: np.ndarray) -> np.ndarray:
    n = np.arange(1, N_BESSEL + 1)
    return np.sqrt(2.0 / R_CUT) * np.sin(n[None, :] * pi * r[:, None] / R_CUT) / r[:, None]


S_CHUNK = 1 << 16   # edges per independently seeded chunk of s


def edge_weights(cfg: Config, vec: np.ndarray, e0: int, e1: int, W=None) -> np.ndarray:
    """Per-edge, per-path, per-channel weights s[e0:e1] as float32 [n, P, C]."""
    P, _ = n_paths_dout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    C = cfg.channels
    if cfg.weights == "bessel":
        if W is None:
            W = bessel_matrix(cfg)
        r = np.linalg.norm(vec[e0:e1].astype(np.float64), axis=1)
        return (bessel_basis(r) @ W).astype(np.float32).reshape(e1 - e0, P, C)
    out = np.empty((e1 - e0, P, C), dtype=np.float32)
    c0 = e0 // S_CHUNK
    c1 = (e1 - 1) // S_CHUNK if e1 > e0 else c0 - 1
    for c in range(c0, c1 + 1):
        lo, hi = c * S_CHUNK, (c + 1) * S_CHUNK
        blk = normal_f32(cfg.cid, _S, (S_CHUNK, P, C), chunk=c)
        a, b = max(lo, e0), min(hi, e1)
        out[a - e0:b - e0] = blk[a - lo:b - lo]
    return out


def edge_weights_rows(cfg: Config, vec: np.ndarray, rows: np.ndarray, W=None) -> np.ndarray:
    """s for an arbitrary set of edge ids (regenerates only the chunks needed)."""
    rows = np.asarray(rows, dtype=np.int64)
    P, _ = n_paths_dout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    out = np.empty((rows.shape[0], P, cfg.channels), dtype=np.float32)
    if cfg.weights == "bessel":
        if W is None:
            W = bessel_matrix(cfg)
        r = np.linalg.norm(vec[rows].astype(np.float64), axis=1)
        return (bessel_basis(r) @ W).astype(np.float32).reshape(rows.shape[0], P, cfg.channels)
    for c in np.unique(rows // S_CHUNK):
        sel = np.nonzero(rows // S_CHUNK == c)[0]
        blk = normal_f32(cfg.cid, _S, (S_CHUNK, P, cfg.channels), chunk=int(c))
        out[sel] = blk[rows[sel] - c * S_CHUNK]
    return out


def radial_inputs(cfg: Config, vec: np.ndarray):
    """(h [E, 8], W [8, P, C]) float32 with h = the Bessel basis of |r| and W the
    workload's fixed random matrix: h @ W is its per-edge weight recipe."""
    P, _ = n_paths_dout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    r = np.linalg.norm(vec.astype(np.float64), axis=1)
    h = bessel_basis(r).astype(np.float32)
    W = bessel_matrix(cfg).astype(np.float32).reshape(N_BESSEL, P, cfg.channels)
    return h, W


def tp_inputs(cfg: Config, rows: int | None = None):
    """(x [R, D_in, C], unit vectors u [R, 3], w [R, P, C]) for the tensor product."""
    R = cfg.rows if rows is None else rows
    d_in, C = irreps_dims(cfg.irreps)
    P, _ = n_paths_dout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    x = normal_f32(cfg.cid, _X, (R, d_in, C))
    g = rng(cfg.cid, _VEC).standard_normal((R, 3))
    u = (g / np.linalg.norm(g, axis=1, keepdims=True)).astype(np.float32)
    w = normal_f32(cfg.cid, _S, (R, P, C))
    return x, u, w


def normal_device(cid: int, stream: int, shape, device, chunk_rows: int = 1 << 16):
    """N(0,1) float32 tensor drawn on the device by torch's seeded generator
    (Philox), chunk by chunk along the first axis; for arrays too large to
    draw on the host.  Deterministic for a given (cid, stream, shape)."""
    import torch
    out = torch.empty(shape, dtype=torch.float32, device=device)
    g = torch.Generator(device=device)
    for i, r0 in enumerate(range(0, shape[0], chunk_rows)):
        r1 = min(shape[0], r0 + chunk_rows)
        g.manual_seed(((cid * 1000003 + stream) * 1000003 + i) & 0x7FFFFFFFFFFFFFFF)
        out[r0:r1].normal_(generator=g)
    return out
