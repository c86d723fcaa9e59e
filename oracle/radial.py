"""Radial edge weights produced by a linear layer, fused into the
convolution (oracle side).

Part of the test-only fp64 oracle; see the package docstring.

The per-edge scalars of eq. (message-passing-linear) depend on the edge
length through a radial embedding followed by an MLP (App. A.3, the linear
mixing and message-passing items).  With h_e in R^K the per-edge features
entering the MLP's last linear layer (for a one-layer model: the radial basis
itself) and W in R^{K x P x C} that layer's weight,
    s_e^{k,q} = sum_j h_e^j W^{j,k,q},
and the convolution of eq. (message_passing_convolution) takes these s.
Cotangents, from the ds of eq. (conv-bwd) by the chain rule:
    dW^{j,k,q} = sum_e h_e^j ds_e^{k,q},     dh_e^j = sum_{k,q} ds_e^{k,q} W^{j,k,q}.
einsum is the only library primitive.
"""
from __future__ import annotations

import torch

from . import conv as _conv
from .tp import t64


def weights(h, W) -> torch.Tensor:
    """s [E, P, C] = h [E, K] contracted with W [K, P, C]."""
    return torch.einsum("ej,jkq->ekq", t64(h), t64(W))


def conv_fwd(lay, x, vec, h, W, sender, receiver, n_nodes, pad_node=-1, receivers=None):
    """m [len(receivers) or N, D_out, C] float64."""
    return _conv.conv_fwd(lay, x, vec, weights(h, W), sender, receiver, n_nodes, pad_node, receivers)


def conv_bwd(lay, x, vec, h, W, dm, sender, receiver, n_nodes, pad_node=-1, senders=None, edges=None):
    """Cotangents: dict(dx, dvec, dh, ds, and dW when all edges are requested).

    dh and ds cover the requested edges (all by default); dvec is the harmonic
    part only (the chain through h belongs to whoever computed h)."""
    h = t64(h)
    res = _conv.conv_bwd(lay, x, vec, weights(h, W), dm, sender, receiver, n_nodes, pad_node,
                         senders=senders, edges=edges)
    ds = res["ds"]
    out = dict(dx=res["dx"], dvec=res["dvec"], ds=ds,
               dh=torch.einsum("ekq,jkq->ej", ds, t64(W)))
    if edges is None:
        out["dW"] = torch.einsum("ej,ekq->jkq", h, ds)
    return out
