"""Equivariant linear mixing of irreps features (oracle side).

Part of the test-only fp64 oracle; see the package docstring.

App. A.3 ("Linear mixing") mixes channels and multiplicities linearly between
irreducible features of the same degree.  Written per output irrep: an output
block o of type (l, p) receives every input block of the same (l, p), in input
order, with their multiplicities concatenated ("uvw"), through one matrix
W_o [n_in(o) * C_in, C_out] shared by the 2l+1 components m (a weight that
depended on m would break equivariance):
    out[n, o_row + m, j] = sum_t sum_k x[n, in_row(t) + m, k] W_o[t * C_in + k, j].
An output block with no input of its type is zero.  W is the concatenation of
the W_o in output order.  Backward:
    dx[n, in_row(t) + m, k] = sum_j dout[n, o_row + m, j] W_o[t * C_in + k, j],
    dW_o[t * C_in + k, j]   = sum_{n, m} x[n, in_row(t) + m, k] dout[n, o_row + m, j].
einsum is the only library primitive.
"""
from __future__ import annotations

import numpy as np
import torch

from . import irreps as _ir
from .tp import t64


def blocks(irreps: str):
    """[(l, p, first row, multiplicity)] and the total row count D."""
    out, row = [], 0
    for b in _ir.parse(irreps):
        out.append((b.l, b.p, row, b.mul))
        row += 2 * b.l + 1
    return out, row


def plan(irreps_in: str, irreps_out: str):
    """Per output block: (l, out row, [input rows], offset of W_o in W, size of W_o)."""
    ins, d_in = blocks(irreps_in)
    outs, d_out = blocks(irreps_out)
    c_in, c_out = ins[0][3], outs[0][3]
    res, off = [], 0
    for (l, p, orow, _) in outs:
        src = [irow for (li, pi, irow, _) in ins if (li, pi) == (l, p)]
        n = len(src) * c_in * c_out
        res.append((l, orow, src, off, n))
        off += n
    return res, d_in, d_out, c_in, c_out, off


def forward(irreps_in, irreps_out, x, W):
    x, W = t64(x), t64(W)
    jobs, d_in, d_out, c_in, c_out, _ = plan(irreps_in, irreps_out)
    out = x.new_zeros((x.shape[0], d_out, c_out))
    for l, orow, src, off, n in jobs:
        if not src:
            continue
        Wo = W[off:off + n].reshape(len(src) * c_in, c_out)
        xs = torch.cat([x[:, r:r + 2 * l + 1, :] for r in src], dim=2)   # [N, 2l+1, n_in * C_in]
        out[:, orow:orow + 2 * l + 1, :] = torch.einsum("nmk,kj->nmj", xs, Wo)
    return out


def backward(irreps_in, irreps_out, x, W, dout):
    """(dx, dW) in float64."""
    x, W, dout = t64(x), t64(W), t64(dout)
    jobs, d_in, d_out, c_in, c_out, _ = plan(irreps_in, irreps_out)
    dx = torch.zeros_like(x)
    dW = torch.zeros_like(W)
    for l, orow, src, off, n in jobs:
        if not src:
            continue
        Wo = W[off:off + n].reshape(len(src) * c_in, c_out)
        g = dout[:, orow:orow + 2 * l + 1, :]
        for t, r in enumerate(src):
            dx[:, r:r + 2 * l + 1, :] += torch.einsum("nmj,kj->nmk", g, Wo[t * c_in:(t + 1) * c_in])
            dW[off + t * c_in * c_out:off + (t + 1) * c_in * c_out] = torch.einsum(
                "nmk,nmj->kj", x[:, r:r + 2 * l + 1, :], g).reshape(-1)
    return dx, dW
