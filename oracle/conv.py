"""Message-passing convolution and its cotangents (oracle side).

Part of the test-only fp64 oracle; see the package docstring.

Forward, App. E.1 eq. (message-passing) / (message_passing_convolution):
    m_b^{i0,q} = sum_{a~b} sum_{i1,i2} C^{i0}_{i1,i2} x_a^{i1,q} y_ab^{i2} s_ab^{i3(i0),q}
with y_ab = Y(r_ab/|r_ab|) the real harmonics of the edge vector.

Backward, App. E.1 eq. (conv-bwd), with z_ab = x_a (x) y_ab:
    dx_a  = sum_{b~a} s_ab . (y_ab (x) dm_b)      (transposed coupling)
    dy_ab = s_ab . (x_a (x) dm_b)                 (reduced over channels)
    ds_ab^{(k)} = sum_{M in block k} z_ab^{M} dm_b^{M}
and dvec = J^T dy with J the Jacobian of r -> Y(r/|r|).

Written as plain sums over edges, path by path, with dense per-path coupling
blocks and einsum/index_add as the only library primitives.  Every function
can work on a subset (sampled receivers, senders or edges) so that large
graphs can be checked point by point.  Padding edges (sender or receiver ==
pad_node) contribute nothing and get zero cotangents.
"""
from __future__ import annotations

import numpy as np
import torch

from . import cg as _cg
from . import sh as _sh
from .tp import t64


def _np(a):
    if isinstance(a, torch.Tensor):
        return a.detach().cpu().numpy()
    return np.asarray(a)


def _blocks(lay):
    return [torch.as_tensor(b) for b in _cg.path_blocks(lay)]


def edge_messages(lay, xs, y, s) -> torch.Tensor:
    """m~_e = s_e . (x_send(e) (x) y_e) for a batch of edges, float64."""
    E, _, C = xs.shape
    out = xs.new_zeros((E, lay.d_out, C))
    for p, blk in zip(lay.paths, _blocks(lay)):
        xb = xs[:, p.x_off:p.x_off + 2 * p.l1 + 1, :]
        yb = y[:, p.y_off:p.y_off + 2 * p.l2 + 1]
        z = torch.einsum("Mab,eaq,eb->eMq", blk, xb, yb)
        out[:, p.out_off:p.out_off + 2 * p.l3 + 1, :] = z * s[:, p.k, None, :]
    return out


def conv_fwd_from_y(lay, x, y, s, sender, receiver, n_nodes, pad_node=-1,
                    receivers=None, chunk=2048):
    """Forward with the harmonics y [E, D_sh] given; differentiable in x, y, s."""
    x, y, s = t64(x), t64(y), t64(s)
    snd = _np(sender).astype(np.int64)
    rcv = _np(receiver).astype(np.int64)
    keep = np.ones(snd.shape[0], dtype=bool)
    if pad_node >= 0:
        keep &= (snd != pad_node) & (rcv != pad_node)
    if receivers is None:
        rows = np.arange(n_nodes, dtype=np.int64)
    else:
        rows = np.asarray(receivers, dtype=np.int64)
    where = np.full(n_nodes, -1, dtype=np.int64)
    where[rows] = np.arange(rows.shape[0])
    keep &= where[rcv] >= 0
    eids = np.nonzero(keep)[0]
    C = x.shape[2]
    out = x.new_zeros((rows.shape[0], lay.d_out, C))
    for c0 in range(0, eids.shape[0], chunk):
        e = torch.as_tensor(eids[c0:c0 + chunk])
        msg = edge_messages(lay, x[torch.as_tensor(snd)[e]], y[e], s[e])
        out = out.index_add(0, torch.as_tensor(where[rcv[eids[c0:c0 + chunk]]]), msg)
    return out


def conv_fwd(lay, x, vec, s, sender, receiver, n_nodes, pad_node=-1, receivers=None,
             chunk=2048):
    """m [len(receivers) or N, D_out, C] float64."""
    vec = t64(vec)
    y = _sh.sh_vec(lay.lmax_sh, vec)
    return conv_fwd_from_y(lay, x, y, s, sender, receiver, n_nodes, pad_node,
                           receivers, chunk)


def conv_bwd_from_y(lay, x, y, s, dm, sender, receiver, n_nodes, pad_node=-1,
                    senders=None, edges=None, chunk=1024):
    """Cotangents of eq. (conv-bwd) with the harmonics y [E, D_sh] given.

    Returns dict(dx=[len(senders) or N, D_in, C], ds=[len(edges) or E, P, C],
    dy=[len(edges) or E, D_sh]), all float64; differentiable in x, y, s, dm.
    """
    x, y, s, dm = t64(x), t64(y), t64(s), t64(dm)
    snd = _np(sender).astype(np.int64)
    rcv = _np(receiver).astype(np.int64)
    E = snd.shape[0]
    keep = np.ones(E, dtype=bool)
    if pad_node >= 0:
        keep &= (snd != pad_node) & (rcv != pad_node)
    C = x.shape[2]
    blocks = _blocks(lay)

    # --- dx: sum over out-edges of each requested sender -------------------
    srows = np.arange(n_nodes, dtype=np.int64) if senders is None else np.asarray(senders, np.int64)
    where = np.full(n_nodes, -1, dtype=np.int64)
    where[srows] = np.arange(srows.shape[0])
    eids = np.nonzero(keep & (where[snd] >= 0))[0]
    dx = x.new_zeros((srows.shape[0], lay.d_in, C))
    for c0 in range(0, eids.shape[0], chunk):
        e = eids[c0:c0 + chunk]
        ye = y[torch.as_tensor(e)]
        se = s[torch.as_tensor(e)]
        dmb = dm[torch.as_tensor(rcv[e])]
        t = x.new_zeros((e.shape[0], lay.d_in, C))
        for p, blk in zip(lay.paths, blocks):
            yb = ye[:, p.y_off:p.y_off + 2 * p.l2 + 1]
            dmk = dmb[:, p.out_off:p.out_off + 2 * p.l3 + 1, :]
            t[:, p.x_off:p.x_off + 2 * p.l1 + 1, :] += torch.einsum(
                "Mab,eb,eq,eMq->eaq", blk, yb, se[:, p.k, :], dmk)
        dx = dx.index_add(0, torch.as_tensor(where[snd[e]]), t)

    # --- ds, dy: edge-local ------------------------------------------------
    erows = np.arange(E, dtype=np.int64) if edges is None else np.asarray(edges, np.int64)
    ds = x.new_zeros((erows.shape[0], lay.n_paths, C))
    dy = x.new_zeros((erows.shape[0], lay.d_sh))
    live = np.nonzero(keep[erows])[0]
    for c0 in range(0, live.shape[0], chunk):
        pos = live[c0:c0 + chunk]
        e = erows[pos]
        et = torch.as_tensor(e)
        ye = y[et]
        xa = x[torch.as_tensor(snd[e])]
        se = s[et]
        dmb = dm[torch.as_tensor(rcv[e])]
        dsc = x.new_zeros((e.shape[0], lay.n_paths, C))
        dyc = x.new_zeros((e.shape[0], lay.d_sh))
        for p, blk in zip(lay.paths, blocks):
            xb = xa[:, p.x_off:p.x_off + 2 * p.l1 + 1, :]
            yb = ye[:, p.y_off:p.y_off + 2 * p.l2 + 1]
            dmk = dmb[:, p.out_off:p.out_off + 2 * p.l3 + 1, :]
            z = torch.einsum("Mab,eaq,eb->eMq", blk, xb, yb)
            dsc[:, p.k, :] = (z * dmk).sum(dim=1)
            dyc[:, p.y_off:p.y_off + 2 * p.l2 + 1] += torch.einsum(
                "Mab,eaq,eMq,eq->eb", blk, xb, dmk, se[:, p.k, :])
        ds = ds.index_put((torch.as_tensor(pos),), dsc)
        dy = dy.index_put((torch.as_tensor(pos),), dyc)
    return dict(dx=dx, ds=ds, dy=dy)


def conv_bwd(lay, x, vec, s, dm, sender, receiver, n_nodes, pad_node=-1,
             senders=None, edges=None, chunk=1024):
    """Cotangents of eq. (conv-bwd) for y = Y(vec), plus dvec = J^T dy.

    Returns dict(dx=[len(senders) or N, D_in, C], ds=[len(edges) or E, P, C],
    dvec=[len(edges) or E, 3], dy=[len(edges) or E, D_sh]), all float64.
    """
    vec = t64(vec)
    y = _sh.sh_vec(lay.lmax_sh, vec)
    res = conv_bwd_from_y(lay, x, y, s, dm, sender, receiver, n_nodes, pad_node, senders, edges, chunk)
    erows = np.arange(vec.shape[0], dtype=np.int64) if edges is None else np.asarray(edges, np.int64)
    snd = _np(sender).astype(np.int64)
    rcv = _np(receiver).astype(np.int64)
    live = np.ones(erows.shape[0], dtype=bool)
    if pad_node >= 0:
        live &= (snd[erows] != pad_node) & (rcv[erows] != pad_node)
    dvec = vec.new_zeros((erows.shape[0], 3))
    idx = np.nonzero(live)[0]
    if idx.shape[0]:
        dvec[torch.as_tensor(idx)] = _sh.sh_vec_vjp(lay.lmax_sh, vec[torch.as_tensor(erows[idx])],
                                                    res["dy"][torch.as_tensor(idx)])
    res["dvec"] = dvec
    return res


def conv_bwd2(lay, x, y, s, dm, ddx, ddy, dds, sender, receiver, n_nodes, pad_node=-1):
    """Second-order rule of eq. (conv-bwd-bwd-ddm) and eq. (conv-bwd2-xys).

    (ddx, ddy, dds) are variations of the backward's outputs (dx, dy, ds); the
    result holds the variations of its inputs: dict(dx, dy, ds, ddm), with
        ddm = conv(ddx, y, s) + conv(x, ddy, s) + conv(x, y, dds)
        dx  = dx of conv_bwd(x, ddy, s, dm) + dx of conv_bwd(x, y, dds, dm)
        dy  = dy of conv_bwd(ddx, y, s, dm) + dy of conv_bwd(x, y, dds, dm)
        ds  = ds of conv_bwd(ddx, y, s, dm) + ds of conv_bwd(x, ddy, s, dm).
    """
    def f(a, b, c):
        return conv_fwd_from_y(lay, a, b, c, sender, receiver, n_nodes, pad_node)

    def b(a, yy, c):
        return conv_bwd_from_y(lay, a, yy, c, dm, sender, receiver, n_nodes, pad_node)

    ddm = f(ddx, y, s) + f(x, ddy, s) + f(x, y, dds)
    bx, by, bs = b(ddx, y, s), b(x, ddy, s), b(x, y, dds)
    return dict(dx=by["dx"] + bs["dx"], dy=bx["dy"] + bs["dy"], ds=bx["ds"] + by["ds"], ddm=ddm)
