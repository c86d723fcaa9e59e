"""Helpers for the GPU parity tests: upload seeded inputs, build compact
sub-problems the fp64 oracle can solve for sampled rows, and compare."""
from __future__ import annotations

import numpy as np

import synth
from oracle import conv as oconv
from oracle import irreps as oirreps

TOL = 1e-5   # relative L2 per output tensor, float32 path vs float64 oracle


def rel_l2(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def to_np(t):
    return t.detach().cpu().numpy()


def upload_weights(cfg, vec: np.ndarray, chunk: int = 1 << 16):
    """s for every edge, generated on the host chunk by chunk and copied up."""
    import torch
    E = vec.shape[0]
    P, _ = synth.n_paths_dout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    s = torch.empty((E, P, cfg.channels), dtype=torch.float32, device="cuda")
    W = synth.bessel_matrix(cfg) if cfg.weights == "bessel" else None
    for e0 in range(0, E, chunk):
        e1 = min(E, e0 + chunk)
        s[e0:e1].copy_(torch.from_numpy(synth.edge_weights(cfg, vec, e0, e1, W=W)))
    return s


def _rows(a, idx):
    """Rows of a host array or (sampled) of a device tensor, as numpy."""
    if isinstance(a, np.ndarray):
        return a[idx]
    import torch
    return a[torch.as_tensor(np.asarray(idx), device=a.device)].cpu().numpy()


def _compact(snd, rcv, sel):
    """Renumber the nodes touched by edges sel to 0..k-1 (sub-problem for the oracle)."""
    nodes, inv = np.unique(np.concatenate([snd[sel], rcv[sel]]), return_inverse=True)
    k = sel.shape[0]
    return nodes, inv[:k], inv[k:]


def oracle_fwd_rows(lay, x, vec, s_rows_fn, snd, rcv, n_nodes, receivers, pad=-1):
    """m for the given receivers, using only their in-edges (x: host array or
    device tensor; only the rows the sub-problem touches are read)."""
    assert pad < 0, "sampled checks run on graphs without padding"
    receivers = np.asarray(receivers, dtype=np.int64)
    sel = np.nonzero(np.isin(rcv, receivers))[0]
    res = np.zeros((receivers.shape[0], lay.d_out, lay.channels))
    if sel.shape[0] == 0:
        return res
    nodes, sc, rc = _compact(snd, rcv, sel)
    # receivers without in-edges are not in the compact node set: their row stays zero
    present = np.isin(receivers, nodes)
    out = oconv.conv_fwd(lay, _rows(x, nodes), vec[sel], s_rows_fn(sel), sc, rc, nodes.shape[0],
                         receivers=np.searchsorted(nodes, receivers[present]))
    res[present] = out.numpy()
    return res


def oracle_bwd_rows(lay, x, vec, s_rows_fn, dm, snd, rcv, n_nodes, senders, edges, pad=-1):
    """dx for the given senders and ds, dvec for the given edges (x, dm: host
    arrays or device tensors).  Padding edges must not be among them."""
    assert pad < 0, "sampled checks run on graphs without padding"
    senders = np.asarray(senders, dtype=np.int64)
    edges = np.asarray(edges, dtype=np.int64)
    sel = np.nonzero(np.isin(snd, senders))[0]
    dx = np.zeros((senders.shape[0], lay.d_in, lay.channels))
    if sel.shape[0]:
        nodes, sc, rc = _compact(snd, rcv, sel)
        present = np.isin(senders, nodes)
        dx[present] = oconv.conv_bwd(lay, _rows(x, nodes), vec[sel], s_rows_fn(sel), _rows(dm, nodes), sc,
                                     rc, nodes.shape[0], senders=np.searchsorted(nodes, senders[present]),
                                     edges=np.zeros(0, np.int64))["dx"].numpy()
    nodes, sc, rc = _compact(snd, rcv, edges)
    res = oconv.conv_bwd(lay, _rows(x, nodes), vec[edges], s_rows_fn(edges), _rows(dm, nodes), sc, rc,
                         nodes.shape[0], senders=np.zeros(0, np.int64))
    return dx, res["ds"].numpy(), res["dvec"].numpy()


def layout_of(cfg):
    return oirreps.layout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
