"""Receiver- and sender-ordered CSR of an edge list (oracle side).

Part of the test-only fp64 oracle; see the package docstring.

App. E.2.2 and App. E.3 traverse edges through a compressed-sparse-row
structure ordered by receiver; App. E.4 (backward) traverses them ordered by
sender.  Reading adopted: edges with equal key keep their original edge-id
order (a stable sort), which makes the permutation unique.  Padding edges
(sender or receiver equal to the padding node, App. C / the padding discussion
of the results section) are left out of both structures.
"""
from __future__ import annotations

import numpy as np


def csr(key: np.ndarray, n_nodes: int, keep: np.ndarray | None = None):
    """(perm, rowptr): edge ids sorted stably by key, and segment offsets."""
    key = np.asarray(key, dtype=np.int64)
    ids = np.arange(key.shape[0], dtype=np.int64)
    if keep is not None:
        ids = ids[keep]
    perm = ids[np.argsort(key[ids], kind="stable")]
    counts = np.bincount(key[perm], minlength=n_nodes)
    rowptr = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    return perm, rowptr


def not_pad(sender, receiver, pad_node: int) -> np.ndarray:
    sender = np.asarray(sender)
    receiver = np.asarray(receiver)
    if pad_node < 0:
        return np.ones(sender.shape[0], dtype=bool)
    return (sender != pad_node) & (receiver != pad_node)


def build(sender, receiver, n_nodes: int, pad_node: int = -1):
    keep = not_pad(sender, receiver, pad_node)
    perm_r, rowptr_r = csr(receiver, n_nodes, keep)
    perm_s, rowptr_s = csr(sender, n_nodes, keep)
    return perm_r, rowptr_r, perm_s, rowptr_s
