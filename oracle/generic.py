"""Tensor product with caller-supplied coefficient records (oracle side).

Part of the test-only fp64 oracle; see the package docstring.

App. E.2 unfolds the coupling into sparse records (i0, i1, i2, value): the
generic sparse tensor product is
    z[r, i0, q] = sum over records (i0, i1, i2, v) of v x[r, i1, q] y[r, i2(, q)]
with y either per channel or shared by the channels.  Any record set is
allowed (e.g. several paths summed into one output block, App. C's collapsed
output multiplicities).  The backward follows eq. (tp-bwd): the same product
with the records permuted,
    dx = tensor_product(C^{i1}_{i2 i0}, y, dz),   dy = tensor_product(C^{i2}_{i1 i0}, x, dz),
where a shared y collects dy over the channels.  Both directions are written
as explicit loops over the records; no library primitive beyond elementwise
array arithmetic.
"""
from __future__ import annotations

import numpy as np


def tp(i0, i1, i2, val, x, y, d_z):
    """z [R, d_z, C] float64; y [R, d_y, C] (per channel) or [R, d_y] (shared)."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    i0, i1, i2 = (np.asarray(a, np.int64) for a in (i0, i1, i2))
    val = np.asarray(val, np.float64)
    R, _, C = x.shape
    z = np.zeros((R, d_z, C))
    yy = y if y.ndim == 3 else y[:, :, None]
    terms = val[None, :, None] * x[:, i1, :] * yy[:, i2, :]          # [R, nnz, C]
    for k in range(i0.shape[0]):
        z[:, i0[k], :] += terms[:, k, :]
    return z


def tp_bwd(i0, i1, i2, val, x, y, dz):
    """(dx, dy) of tp, as eq. (tp-bwd): the product with permuted records."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    dz = np.asarray(dz, np.float64)
    # per record: dx[i1] += v y[i2] dz[i0] and dy[i2] += v x[i1] dz[i0]
    R, _, C = x.shape
    dx = np.zeros_like(x)
    dy = np.zeros_like(y)
    yy = y if y.ndim == 3 else y[:, :, None]
    for k in range(len(val)):
        a, b, c, v = int(i0[k]), int(i1[k]), int(i2[k]), float(val[k])
        dx[:, b, :] += v * yy[:, c, :] * dz[:, a, :]
        t = v * x[:, b, :] * dz[:, a, :]
        if y.ndim == 3:
            dy[:, c, :] += t
        else:
            dy[:, c] += t.sum(axis=1)
    return dx, dy
