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


def oracle_fwd_rows(lay, x, vec, s_rows_fn, snd, rcv, n_nodes, receivers, pad=-1):
    """m for the given receivers, using only their in-edges."""
    receivers = np.asarray(receivers, dtype=np.int64)
    sel = np.nonzero(np.isin(rcv, receivers))[0]
    s_sub = s_rows_fn(sel)
    return oconv.conv_fwd(lay, x, vec[sel], s_sub, snd[sel], rcv[sel], n_nodes, pad_node=pad,
                          receivers=receivers).numpy()


def oracle_bwd_rows(lay, x, vec, s_rows_fn, dm, snd, rcv, n_nodes, senders, edges, pad=-1):
    """dx for the given senders and ds, dvec for the given edges."""
    senders = np.asarray(senders, dtype=np.int64)
    edges = np.asarray(edges, dtype=np.int64)
    sel = np.nonzero(np.isin(snd, senders))[0]
    out_dx = oconv.conv_bwd(lay, x, vec[sel], s_rows_fn(sel), dm, snd[sel], rcv[sel], n_nodes,
                            pad_node=pad, senders=senders, edges=np.zeros(0, np.int64))["dx"].numpy()
    res = oconv.conv_bwd(lay, x, vec[edges], s_rows_fn(edges), dm, snd[edges], rcv[edges], n_nodes,
                         pad_node=pad, senders=np.zeros(0, np.int64))
    return out_dx, res["ds"].numpy(), res["dvec"].numpy()


def layout_of(cfg):
    return oirreps.layout(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
