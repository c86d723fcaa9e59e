"""Channelwise weighted tensor product (oracle side).

Part of the test-only fp64 oracle; see the package docstring.

Follows App. E.1, eq. (tensor_product_formula)
    z^{i0,q} = sum_{i1,i2} C^{i0}_{i1,i2} x^{i1,q} y^{i2,q}
and eq. (edge_scalar_weighting)
    m^{i0,q} = z^{i0,q} s^{i3(i0),q}.
The harmonics y carry no channel axis here: they are broadcast over the
channels (the convolution algorithms of App. E.3 take y in R^{E x d'}).

Written path by path with the dense real coupling block of each path; the
only library primitive is einsum.
"""
from __future__ import annotations

import numpy as np
import torch

from . import cg as _cg


def t64(a) -> torch.Tensor:
    if isinstance(a, torch.Tensor):
        return a.to(torch.float64)
    return torch.as_tensor(np.asarray(a), dtype=torch.float64)


def _blocks(lay):
    return [torch.as_tensor(b) for b in _cg.path_blocks(lay)]


def tp_unweighted(lay, x, y) -> torch.Tensor:
    """z[r, i0, q] = sum C x[r, i1, q] y[r, i2]  (eq. tensor_product_formula)."""
    x, y = t64(x), t64(y)
    R, _, C = x.shape
    z = x.new_zeros((R, lay.d_out, C))
    for p, blk in zip(lay.paths, _blocks(lay)):
        xb = x[:, p.x_off:p.x_off + 2 * p.l1 + 1, :]
        yb = y[:, p.y_off:p.y_off + 2 * p.l2 + 1]
        z[:, p.out_off:p.out_off + 2 * p.l3 + 1, :] = torch.einsum("Mab,raq,rb->rMq", blk, xb, yb)
    return z


def weight(lay, z, w) -> torch.Tensor:
    """m[r, i0, q] = z[r, i0, q] * w[r, i3(i0), q]  (eq. edge_scalar_weighting)."""
    z, w = t64(z), t64(w)
    idx = torch.as_tensor(lay.i3(), dtype=torch.long)
    return z * w[:, idx, :]


def tp(lay, x, y, w) -> torch.Tensor:
    """Weighted tensor product, float64 [R, D_out, C]."""
    return weight(lay, tp_unweighted(lay, x, y), w)


def tp_bwd(lay, x, y, w, dz):
    """Cotangents of the weighted tensor product (App. E.1, eq. tp-bwd, with
    the path weight of eq. edge_scalar_weighting):
        dw[r,k,q]  = sum_{M in k} dz[r,M,q] * (x (x) y)[r,M,q]
        dx[r,i1,q] = sum_{i0,i2} C[i0,i1,i2] y[r,i2] w[r,i3(i0),q] dz[r,i0,q]
        dy[r,i2]   = sum_q sum_{i0,i1} C[i0,i1,i2] x[r,i1,q] w[r,i3(i0),q] dz[r,i0,q]
    Returns (dx, dy, dw) in float64."""
    x, y, w, dz = t64(x), t64(y), t64(w), t64(dz)
    R, _, C = x.shape
    dx = torch.zeros_like(x)
    dy = torch.zeros_like(y)
    dw = torch.zeros_like(w)
    for p, blk in zip(lay.paths, _blocks(lay)):
        xb = x[:, p.x_off:p.x_off + 2 * p.l1 + 1, :]
        yb = y[:, p.y_off:p.y_off + 2 * p.l2 + 1]
        dzb = dz[:, p.out_off:p.out_off + 2 * p.l3 + 1, :]
        wk = w[:, p.k, :]
        u = torch.einsum("Mab,raq,rb->rMq", blk, xb, yb)
        dw[:, p.k, :] = (u * dzb).sum(dim=1)
        dx[:, p.x_off:p.x_off + 2 * p.l1 + 1, :] += torch.einsum("Mab,rb,rq,rMq->raq", blk, yb, wk, dzb)
        dy[:, p.y_off:p.y_off + 2 * p.l2 + 1] += torch.einsum("Mab,raq,rq,rMq->rb", blk, xb, wk, dzb)
    return dx, dy, dw
