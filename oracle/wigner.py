"""Wigner-D matrices of the real harmonics (tests only).

Part of the test-only fp64 oracle; see the package docstring.

App. A.2 ("Equivariance"): for every rotation g there is a matrix D_g with
Y_l(g u) = D_g Y_l(u).  Here D_l(R) is obtained as the least-squares solution
of that identity over random sample points; it does not use the coupling
tables, so it can test them.
"""
from __future__ import annotations

import numpy as np

from . import sh as _sh


def random_rotation(rng) -> np.ndarray:
    """Uniform random rotation from a normalised Gaussian quaternion."""
    q = rng.standard_normal(4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([
        [1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)],
    ])


def wigner_d(l: int, R: np.ndarray, seed: int = 7) -> np.ndarray:
    rng = np.random.default_rng(seed + 31 * l)
    g = rng.standard_normal((6 * (2 * l + 1) + 16, 3))
    u = g / np.linalg.norm(g, axis=1, keepdims=True)
    Y = _sh.sh_unit(l, u)[:, l * l:]            # [K, 2l+1]
    YR = _sh.sh_unit(l, u @ R.T)[:, l * l:]     # Y(R u)
    # YR = Y @ D^T
    dt, *_ = np.linalg.lstsq(Y, YR, rcond=None)
    return dt.T
