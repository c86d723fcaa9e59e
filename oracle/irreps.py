"""Irreps descriptors and the list of channelwise coupling paths (oracle side).

Part of the test-only fp64 oracle; see the package docstring.

Follows:
  * App. A.3, "Tensor product": a degree-l1 feature coupled with a degree-l2
    harmonic produces output degrees L = |l1-l2| ... l1+l2.
  * App. B.1: the parity of a path's output is the product of the input
    parities (p1 * p2 = p3).
  * App. E.1, eq. (edge_scalar_weighting): the map i3 sends each output
    coordinate to the scalar block (the path) it belongs to; it is fixed when
    the coefficients are built.

Readings adopted where the paper is silent:
  * every x block carries the same multiplicity C (channelwise / "uvu");
  * harmonic blocks are l2 = 0..lmax_sh with parity (-1)^l2;
  * paths are enumerated x block (in the given order), then l2 ascending, then
    l3 ascending, keeping l3 <= lmax_out; every triangle-allowed path is kept
    whatever its output parity ("all" parities), or only those whose output
    parity is (-1)^l3 ("natural");
  * output blocks are laid out in path order, no sorting by degree.
"""
from __future__ import annotations

import re
from dataclasses import dataclass


@dataclass(frozen=True)
class Block:
    mul: int
    l: int
    p: int  # +1 even, -1 odd


@dataclass(frozen=True)
class Path:
    k: int       # path index == scalar block index (i3 value)
    xb: int      # index of the x block
    l1: int
    p1: int
    l2: int
    l3: int
    p3: int
    x_off: int   # first row of the x block in the D_in axis
    y_off: int   # first row of the harmonic block in the D_sh axis (l2*l2)
    out_off: int  # first row of the output block in the D_out axis


_TOKEN = re.compile(r"^\s*(?:(\d+)\s*x\s*)?(\d+)\s*([eo])\s*$")


def parse(irreps: str) -> list[Block]:
    """Parse "8x0e+8x1o" (multiplicity defaults to 1)."""
    if not isinstance(irreps, str) or not irreps.strip():
        raise ValueError("empty irreps string")
    out = []
    for tok in irreps.split("+"):
        m = _TOKEN.match(tok)
        if m is None:
            raise ValueError(f"bad irreps token {tok!r}")
        mul = int(m.group(1)) if m.group(1) is not None else 1
        l = int(m.group(2))
        p = 1 if m.group(3) == "e" else -1
        if mul <= 0:
            raise ValueError("multiplicity must be positive")
        out.append(Block(mul, l, p))
    return out


@dataclass(frozen=True)
class Layout:
    blocks: tuple
    channels: int
    lmax_sh: int
    lmax_out: int
    paths: tuple
    d_in: int
    d_sh: int
    d_out: int

    @property
    def n_paths(self) -> int:
        return len(self.paths)

    def i3(self):
        """Map output coordinate -> path index (the map i3 of App. E.1)."""
        res = []
        for p in self.paths:
            res += [p.k] * (2 * p.l3 + 1)
        return res


def layout(irreps: str, lmax_sh: int, lmax_out: int, parity: str = "all") -> Layout:
    blocks = parse(irreps)
    muls = {b.mul for b in blocks}
    if len(muls) != 1:
        raise ValueError("channelwise coupling needs one multiplicity for every block")
    if parity not in ("all", "natural"):
        raise ValueError("parity must be 'all' or 'natural'")
    if lmax_sh < 0 or lmax_out < 0:
        raise ValueError("negative degree")
    C = muls.pop()
    x_offs = []
    off = 0
    for b in blocks:
        x_offs.append(off)
        off += 2 * b.l + 1
    d_in = off
    paths = []
    out_off = 0
    for xb, b in enumerate(blocks):
        for l2 in range(lmax_sh + 1):
            p2 = (-1) ** l2
            for l3 in range(abs(b.l - l2), min(b.l + l2, lmax_out) + 1):
                p3 = b.p * p2
                if parity == "natural" and p3 != (-1) ** l3:
                    continue
                paths.append(Path(len(paths), xb, b.l, b.p, l2, l3, p3,
                                  x_offs[xb], l2 * l2, out_off))
                out_off += 2 * l3 + 1
    return Layout(tuple(blocks), C, lmax_sh, lmax_out, tuple(paths), d_in,
                  (lmax_sh + 1) ** 2, out_off)
