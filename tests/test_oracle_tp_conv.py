"""Pins of the oracle's tensor product, convolution and backward.

Each check compares against something the oracle's own formula does not
produce: a brute-force dense contraction, an explicit per-edge loop, float64
autograd of the forward, central finite differences, rotation/inversion
symmetry, and the trilinear (Euler) identity.
"""
import numpy as np
import pytest
import torch

from oracle import cg, conv, graph, irreps, sh, tp, wigner


def _unit(rng, n):
    g = rng.standard_normal((n, 3))
    return g / np.linalg.norm(g, axis=1, keepdims=True)


def _small_graph(rng, n=9, e=40, pad=-1):
    snd = rng.integers(0, n, e)
    rcv = rng.integers(0, n, e)
    rcv = np.where(rcv == snd, (rcv + 1) % n, rcv)
    vec = rng.standard_normal((e, 3)) * 1.7
    return snd.astype(np.int32), rcv.astype(np.int32), vec


LAYS = [("2x0e+2x1o", 2, 2), ("3x0e+3x1o+3x2e", 3, 3), ("2x0e+2x1o+2x2e+2x3o", 3, 3),
        ("2x1e+2x0o", 2, 1)]


@pytest.mark.parametrize("spec", LAYS)
def test_tp_equals_dense_bruteforce(spec):
    lay = irreps.layout(*spec)
    rng = np.random.default_rng(10)
    R, C = 7, lay.channels
    x = rng.standard_normal((R, lay.d_in, C))
    y = sh.sh_unit(lay.lmax_sh, _unit(rng, R))
    w = rng.standard_normal((R, lay.n_paths, C))
    T = cg.dense_tensor(lay)                                   # [D_out, D_in, D_sh]
    i3 = np.array(lay.i3())
    ref = np.einsum("oij,riq,rj->roq", T, x, y) * w[:, i3, :]
    got = tp.tp(lay, x, y, w).numpy()
    assert np.abs(got - ref).max() < 1e-13


def test_tp_scalar_path_and_bilinearity():
    lay = irreps.layout("2x0e+2x1o+2x2e", 3, 3)
    rng = np.random.default_rng(11)
    R, C = 5, 2
    x = rng.standard_normal((R, lay.d_in, C))
    y = sh.sh_unit(3, _unit(rng, R))
    w = rng.standard_normal((R, lay.n_paths, C))
    z = tp.tp(lay, x, y, w).numpy()
    for p in lay.paths:
        if p.l1 == 0:   # 0 x l2 -> l2 is the identity coupling: z = w x_0 Y_l2
            ref = w[:, p.k, None, :] * x[:, p.x_off, None, :] * y[:, p.y_off:p.y_off + 2 * p.l2 + 1, None]
            assert np.abs(z[:, p.out_off:p.out_off + 2 * p.l3 + 1] - ref).max() < 1e-14
    x2 = rng.standard_normal(x.shape)
    a, b = 0.7, -1.3
    lhs = tp.tp(lay, a * x + b * x2, y, w).numpy()
    rhs = a * z + b * tp.tp(lay, x2, y, w).numpy()
    assert np.abs(lhs - rhs).max() < 1e-12


def _rot_features(lay, x, R, out=False):
    """Apply the block-diagonal Wigner-D to the feature axis."""
    x = np.array(x, copy=True)
    if not out:
        for b, off in zip(lay.blocks, _x_offsets(lay)):
            D = wigner.wigner_d(b.l, R)
            x[:, off:off + 2 * b.l + 1] = np.einsum("ij,njq->niq", D, x[:, off:off + 2 * b.l + 1])
    else:
        for p in lay.paths:
            D = wigner.wigner_d(p.l3, R)
            sl = slice(p.out_off, p.out_off + 2 * p.l3 + 1)
            x[:, sl] = np.einsum("ij,njq->niq", D, x[:, sl])
    return x


def _x_offsets(lay):
    offs, o = [], 0
    for b in lay.blocks:
        offs.append(o)
        o += 2 * b.l + 1
    return offs


def test_tp_equivariance():
    lay = irreps.layout("2x0e+2x1o+2x2e+2x3o", 3, 3)
    rng = np.random.default_rng(12)
    R = wigner.random_rotation(rng)
    n, C = 6, 2
    x = rng.standard_normal((n, lay.d_in, C))
    u = _unit(rng, n)
    w = rng.standard_normal((n, lay.n_paths, C))
    z = tp.tp(lay, x, sh.sh_unit(3, u), w).numpy()
    zr = tp.tp(lay, _rot_features(lay, x, R), sh.sh_unit(3, u @ R.T), w).numpy()
    assert np.abs(zr - _rot_features(lay, z, R, out=True)).max() < 1e-11


def _conv_loop(lay, x, vec, s, snd, rcv, n, pad=-1):
    """Materialise every edge message, then scatter with np.add.at."""
    y = sh.sh_vec(lay.lmax_sh, vec)
    T = cg.dense_tensor(lay)
    i3 = np.array(lay.i3())
    out = np.zeros((n, lay.d_out, x.shape[2]))
    for e in range(snd.shape[0]):
        if pad >= 0 and (snd[e] == pad or rcv[e] == pad):
            continue
        msg = np.einsum("oij,iq,j->oq", T, x[snd[e]], y[e]) * s[e][i3]
        np.add.at(out, rcv[e], msg)
    return out


@pytest.mark.parametrize("pad", [-1, 3])
def test_conv_equals_materialised_messages(pad):
    lay = irreps.layout("2x0e+2x1o+2x2e", 2, 2)
    rng = np.random.default_rng(13)
    n = 9
    snd, rcv, vec = _small_graph(rng, n, 50)
    x = rng.standard_normal((n, lay.d_in, 2))
    s = rng.standard_normal((50, lay.n_paths, 2))
    ref = _conv_loop(lay, x, vec, s, snd, rcv, n, pad)
    got = conv.conv_fwd(lay, x, vec, s, snd, rcv, n, pad_node=pad, chunk=7).numpy()
    assert np.abs(got - ref).max() < 1e-12
    # a subset of receivers gives the same rows
    sub = np.array([5, 0, 8])
    part = conv.conv_fwd(lay, x, vec, s, snd, rcv, n, pad_node=pad, receivers=sub).numpy()
    assert np.abs(part - ref[sub]).max() < 1e-12
    if pad >= 0:
        assert np.abs(got[pad]).max() == 0.0


def test_conv_one_in_edge_equals_tp_and_permutation():
    lay = irreps.layout("2x0e+2x1o+2x2e", 3, 3)
    rng = np.random.default_rng(14)
    n = 6
    snd = np.array([3, 4, 5, 0, 1, 2], dtype=np.int32)
    rcv = np.arange(n, dtype=np.int32)
    vec = rng.standard_normal((n, 3))
    x = rng.standard_normal((n, lay.d_in, 2))
    s = rng.standard_normal((n, lay.n_paths, 2))
    m = conv.conv_fwd(lay, x, vec, s, snd, rcv, n).numpy()
    z = tp.tp(lay, x[snd], sh.sh_vec(3, vec), s).numpy()
    assert np.abs(m - z).max() < 1e-13
    # permuting the edge list changes nothing (beyond rounding)
    snd2, rcv2, vec2 = _small_graph(rng, n, 30)
    s2 = rng.standard_normal((30, lay.n_paths, 2))
    perm = rng.permutation(30)
    a = conv.conv_fwd(lay, x, vec2, s2, snd2, rcv2, n).numpy()
    b = conv.conv_fwd(lay, x, vec2[perm], s2[perm], snd2[perm], rcv2[perm], n).numpy()
    assert np.abs(a - b).max() < 1e-12


def test_conv_equivariance_and_inversion():
    lay = irreps.layout("2x0e+2x1o+2x2e+2x3o", 3, 3)
    rng = np.random.default_rng(15)
    n = 8
    snd, rcv, vec = _small_graph(rng, n, 40)
    x = rng.standard_normal((n, lay.d_in, 2))
    s = rng.standard_normal((40, lay.n_paths, 2))
    m = conv.conv_fwd(lay, x, vec, s, snd, rcv, n).numpy()
    R = wigner.random_rotation(rng)
    mr = conv.conv_fwd(lay, _rot_features(lay, x, R), vec @ R.T, s, snd, rcv, n).numpy()
    assert np.abs(mr - _rot_features(lay, m, R, out=True)).max() < 1e-11
    # inversion: r -> -r, x block of parity p -> p x; output block -> p3 * block
    xi = np.array(x)
    for b, off in zip(lay.blocks, _x_offsets(lay)):
        xi[:, off:off + 2 * b.l + 1] *= b.p
    mi = conv.conv_fwd(lay, xi, -vec, s, snd, rcv, n).numpy()
    for p in lay.paths:
        sl = slice(p.out_off, p.out_off + 2 * p.l3 + 1)
        assert np.abs(mi[:, sl] - p.p3 * m[:, sl]).max() < 1e-12


@pytest.mark.parametrize("pad", [-1, 2])
def test_conv_bwd_against_autograd(pad):
    lay = irreps.layout("2x0e+2x1o+2x2e", 3, 3)
    rng = np.random.default_rng(16)
    n, E, C = 7, 35, 3
    snd, rcv, vec = _small_graph(rng, n, E)
    x = torch.tensor(rng.standard_normal((n, lay.d_in, C)), requires_grad=True)
    v = torch.tensor(vec, requires_grad=True)
    s = torch.tensor(rng.standard_normal((E, lay.n_paths, C)), requires_grad=True)
    dm = torch.tensor(rng.standard_normal((n, lay.d_out, C)))
    m = conv.conv_fwd(lay, x, v, s, snd, rcv, n, pad_node=pad)
    gx, gv, gs = torch.autograd.grad(m, (x, v, s), grad_outputs=dm)
    out = conv.conv_bwd(lay, x.detach(), vec, s.detach(), dm, snd, rcv, n, pad_node=pad)
    assert torch.abs(out["dx"] - gx).max() < 1e-12
    assert torch.abs(out["ds"] - gs).max() < 1e-12
    assert torch.abs(out["dvec"] - gv).max() < 1e-11
    # dy against autograd through the harmonics-given forward
    y = sh.sh_vec(3, torch.tensor(vec)).detach().requires_grad_(True)
    m2 = conv.conv_fwd_from_y(lay, x.detach(), y, s.detach(), snd, rcv, n, pad_node=pad)
    gy, = torch.autograd.grad(m2, y, grad_outputs=dm)
    assert torch.abs(out["dy"] - gy).max() < 1e-12
    # sampled outputs equal the full ones
    sub = conv.conv_bwd(lay, x.detach(), vec, s.detach(), dm, snd, rcv, n, pad_node=pad,
                        senders=[4, 1], edges=[0, 9, 33])
    assert torch.abs(sub["dx"] - out["dx"][[4, 1]]).max() < 1e-13
    assert torch.abs(sub["ds"] - out["ds"][[0, 9, 33]]).max() < 1e-13
    assert torch.abs(sub["dvec"] - out["dvec"][[0, 9, 33]]).max() < 1e-13


def test_conv_bwd_finite_differences_and_trilinear_identity():
    lay = irreps.layout("2x0e+2x1o+2x2e+2x3o", 3, 3)
    rng = np.random.default_rng(17)
    n, E, C = 6, 24, 2
    snd, rcv, vec = _small_graph(rng, n, E)
    x = rng.standard_normal((n, lay.d_in, C))
    s = rng.standard_normal((E, lay.n_paths, C))
    dm = rng.standard_normal((n, lay.d_out, C))
    out = conv.conv_bwd(lay, x, vec, s, dm, snd, rcv, n)

    def L(x_, vec_, s_):
        return float((conv.conv_fwd(lay, x_, vec_, s_, snd, rcv, n).numpy() * dm).sum())

    h = 1e-6
    for (a, i, q) in [(0, 3, 1), (4, 12, 0), (5, 0, 1)]:
        xp, xm = x.copy(), x.copy()
        xp[a, i, q] += h
        xm[a, i, q] -= h
        assert abs((L(xp, vec, s) - L(xm, vec, s)) / (2 * h) - out["dx"][a, i, q].item()) < 1e-7
    for (e, k, q) in [(0, 0, 0), (7, 20, 1), (23, 33, 0)]:
        sp, sm = s.copy(), s.copy()
        sp[e, k, q] += h
        sm[e, k, q] -= h
        assert abs((L(x, vec, sp) - L(x, vec, sm)) / (2 * h) - out["ds"][e, k, q].item()) < 1e-7
    for (e, d) in [(1, 0), (11, 2), (19, 1)]:
        vp, vm = vec.copy(), vec.copy()
        vp[e, d] += h
        vm[e, d] -= h
        assert abs((L(x, vp, s) - L(x, vm, s)) / (2 * h) - out["dvec"][e, d].item()) < 1e-6
    # trilinear in (x, y, s): <dm, m> = <dx, x> = <ds, s> = <dy, y>  (Euler)
    m = conv.conv_fwd(lay, x, vec, s, snd, rcv, n).numpy()
    y = sh.sh_vec(3, vec)
    ref = (dm * m).sum()
    for got in [(out["dx"].numpy() * x).sum(), (out["ds"].numpy() * s).sum(),
                (out["dy"].numpy() * y).sum()]:
        assert abs(got - ref) < 1e-10 * max(1.0, abs(ref))
    # dvec is orthogonal to the edge vector (Y is homogeneous of degree 0 in r)
    assert np.abs((out["dvec"].numpy() * vec).sum(1)).max() < 1e-11


def test_graph_csr():
    rng = np.random.default_rng(18)
    n = 11
    snd, rcv, _ = _small_graph(rng, n, 60)
    perm_r, rowptr_r, perm_s, rowptr_s = graph.build(snd, rcv, n, pad_node=4)
    keep = (snd != 4) & (rcv != 4)
    assert rowptr_r[-1] == keep.sum() == perm_r.shape[0]
    assert np.all(np.diff(rowptr_r) >= 0) and np.all(np.diff(rowptr_s) >= 0)
    # brute force: edges of each receiver in increasing edge id
    for b in range(n):
        ids = [e for e in range(60) if rcv[e] == b and keep[e]]
        assert list(perm_r[rowptr_r[b]:rowptr_r[b + 1]]) == ids
        ids = [e for e in range(60) if snd[e] == b and keep[e]]
        assert list(perm_s[rowptr_s[b]:rowptr_s[b + 1]]) == ids


@pytest.mark.parametrize("spec", [("2x0e+2x1o+2x2e", 3, 3), ("3x0e+3x1o+3x2e+3x3o", 3, 3)])
def test_tp_bwd_against_autograd_fd_and_euler(spec):
    lay = irreps.layout(*spec)
    rng = np.random.default_rng(19)
    R, C = 6, lay.channels
    x = torch.tensor(rng.standard_normal((R, lay.d_in, C)), requires_grad=True)
    y = torch.tensor(sh.sh_unit(lay.lmax_sh, _unit(rng, R)), requires_grad=True)
    w = torch.tensor(rng.standard_normal((R, lay.n_paths, C)), requires_grad=True)
    dz = torch.tensor(rng.standard_normal((R, lay.d_out, C)))
    z = tp.tp(lay, x, y, w)
    gx, gy, gw = torch.autograd.grad(z, (x, y, w), grad_outputs=dz)
    dx, dy, dw = tp.tp_bwd(lay, x.detach(), y.detach(), w.detach(), dz)
    assert torch.abs(dx - gx).max() < 1e-12
    assert torch.abs(dy - gy).max() < 1e-12
    assert torch.abs(dw - gw).max() < 1e-12
    # central differences on a few entries
    X, Y, Wt = x.detach().numpy(), y.detach().numpy(), w.detach().numpy()
    L = lambda a, b, c: float((tp.tp(lay, a, b, c).numpy() * dz.numpy()).sum())
    h = 1e-6
    for (r, i, q) in [(0, 1, 0), (5, lay.d_in - 1, C - 1)]:
        a1, a2 = X.copy(), X.copy()
        a1[r, i, q] += h
        a2[r, i, q] -= h
        assert abs((L(a1, Y, Wt) - L(a2, Y, Wt)) / (2 * h) - dx[r, i, q].item()) < 1e-7
    for (r, i) in [(1, 0), (3, lay.d_sh - 1)]:
        b1, b2 = Y.copy(), Y.copy()
        b1[r, i] += h
        b2[r, i] -= h
        assert abs((L(X, b1, Wt) - L(X, b2, Wt)) / (2 * h) - dy[r, i].item()) < 1e-7
    # trilinear: <dz, z> = <dx, x> = <dy, y> = <dw, w>
    ref = float((dz * z.detach()).sum())
    for got in [(dx * x.detach()).sum(), (dy * y.detach()).sum(), (dw * w.detach()).sum()]:
        assert abs(float(got) - ref) < 1e-10 * max(1.0, abs(ref))


# ---------------------------------------------------------------- fused radial weights
def test_radial_one_hot_reduces_to_plain_conv():
    """h_e = unit vector e_j gives s_e = W[j] for every edge."""
    from oracle import radial
    rng = np.random.default_rng(21)
    lay = irreps.layout("2x0e+2x1o+2x2e", 3, 3)
    snd, rcv, vec = _small_graph(rng, n=7, e=25)
    x = rng.standard_normal((7, lay.d_in, lay.channels))
    K = 5
    W = rng.standard_normal((K, lay.n_paths, lay.channels))
    for j in (0, 3):
        h = np.zeros((25, K))
        h[:, j] = 1.0
        ref = conv.conv_fwd(lay, x, vec, np.broadcast_to(W[j], (25,) + W.shape[1:]), snd, rcv, 7)
        got = radial.conv_fwd(lay, x, vec, h, W, snd, rcv, 7)
        assert torch.allclose(got, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("pad", [-1, 4])
def test_radial_bwd_central_differences(pad):
    """<dh, dH> + <dW, dW'> + <dx, dX> equals the directional derivative of
    <dm, m(x, h, W)>, taken by central differences (the loss is trilinear in
    (x, h, W) jointly only through products, so a small step suffices)."""
    from oracle import radial
    rng = np.random.default_rng(22)
    lay = irreps.layout("2x0e+2x1o+2x2e", 2, 2)
    n, e, K = 8, 30, 4
    snd, rcv, vec = _small_graph(rng, n=n, e=e)
    if pad >= 0:
        snd[::7] = pad
    x = rng.standard_normal((n, lay.d_in, lay.channels))
    h = rng.standard_normal((e, K))
    W = rng.standard_normal((K, lay.n_paths, lay.channels))
    dm = rng.standard_normal((n, lay.d_out, lay.channels))
    dX, dH, dW = (rng.standard_normal(a.shape) for a in (x, h, W))
    res = radial.conv_bwd(lay, x, vec, h, W, dm, snd, rcv, n, pad_node=pad)

    def loss(t):
        m = radial.conv_fwd(lay, x + t * dX, vec, h + t * dH, W + t * dW, snd, rcv, n, pad_node=pad)
        return float((m * torch.as_tensor(dm)).sum())

    eps = 1e-3
    fd = (loss(eps) - loss(-eps)) / (2 * eps)
    an = float((res["dx"] * torch.as_tensor(dX)).sum() + (res["dh"] * torch.as_tensor(dH)).sum()
               + (res["dW"] * torch.as_tensor(dW)).sum())
    # the loss is a cubic polynomial in t: central differences carry an eps^2 term only
    assert abs(fd - an) < 1e-5 * max(1.0, abs(an))
    if pad >= 0:
        assert torch.all(res["dh"][snd == pad] == 0)


# ---------------------------------------------------------------- double backward
@pytest.mark.parametrize("spec,pad", [(("2x0e+2x1o+2x2e", 3, 3), -1), (("2x0e+2x1o", 2, 2), 3)])
def test_conv_bwd2_against_autograd_and_central_differences(spec, pad):
    """The composed second-order rule equals (a) float64 autograd of the first
    backward and (b) a five-point difference of L = <ddx, dx> + <ddy, dy> + <dds, ds>
    along a random direction of (x, y, s, dm)."""
    rng = np.random.default_rng(31)
    lay = irreps.layout(*spec)
    n, e = 7, 26
    snd, rcv, vec = _small_graph(rng, n=n, e=e)
    if pad >= 0:
        rcv[::5] = pad
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C))
    y = rng.standard_normal((e, lay.d_sh))          # any y, not only harmonics
    s = rng.standard_normal((e, lay.n_paths, C))
    dm = rng.standard_normal((n, lay.d_out, C))
    ddx = rng.standard_normal(x.shape)
    ddy = rng.standard_normal(y.shape)
    dds = rng.standard_normal(s.shape)
    got = conv.conv_bwd2(lay, x, y, s, dm, ddx, ddy, dds, snd, rcv, n, pad_node=pad)

    def L(xx, yy, ss, mm):
        r = conv.conv_bwd_from_y(lay, xx, yy, ss, mm, snd, rcv, n, pad_node=pad)
        return ((r["dx"] * torch.as_tensor(ddx)).sum() + (r["dy"] * torch.as_tensor(ddy)).sum()
                + (r["ds"] * torch.as_tensor(dds)).sum())

    leaves = [torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (x, y, s, dm)]
    grads = torch.autograd.grad(L(*leaves), leaves)
    for name, g in zip(("dx", "dy", "ds", "ddm"), grads):
        assert torch.allclose(got[name], g, rtol=1e-11, atol=1e-11), name
    u = [rng.standard_normal(a.shape) for a in (x, y, s, dm)]

    def Lt(t):
        return float(L(*[a + t * d for a, d in zip((x, y, s, dm), u)]))

    # L(t) is a cubic in t: the five-point stencil is exact for it up to rounding
    h = 0.1
    fd = (8 * (Lt(h) - Lt(-h)) - (Lt(2 * h) - Lt(-2 * h))) / (12 * h)
    an = sum(float((got[k] * torch.as_tensor(d)).sum()) for k, d in zip(("dx", "dy", "ds", "ddm"), u))
    assert abs(fd - an) < 1e-9 * max(1.0, abs(an))
    if pad >= 0:
        dead = (snd == pad) | (rcv == pad)
        assert torch.all(got["dy"][dead] == 0) and torch.all(got["ds"][dead] == 0)


# ---------------------------------------------------------------- linear mixing
def test_linear_identity_permutation_and_zero_blocks():
    """W_o = identity copies the (single) input block; a permutation matrix
    permutes channels; an output type with no input is zero; two input blocks
    of one type add."""
    from oracle import linear
    rng = np.random.default_rng(41)
    ins, outs = "3x0e+3x1o+3x1o+3x2e", "3x0e+3x1o+3x1e+3x2e"
    jobs, d_in, d_out, c_in, c_out, nw = linear.plan(ins, outs)
    x = rng.standard_normal((5, d_in, 3))
    W = np.zeros(nw)
    perm = np.eye(3)[[2, 0, 1]]
    for l, orow, src, off, n in jobs:
        if l == 0:
            W[off:off + n] = np.eye(3).reshape(-1)
        if l == 1 and src:
            W[off:off + n] = np.concatenate([perm, np.eye(3)]).reshape(-1)
        if l == 2:
            W[off:off + n] = perm.reshape(-1)
    y = linear.forward(ins, outs, x, W).numpy()
    assert np.array_equal(y[:, 0:1], x[:, 0:1])                                   # 0e copied
    assert np.allclose(y[:, 1:4], x[:, 1:4] @ perm + x[:, 4:7], atol=1e-14)        # two 1o blocks
    assert np.all(y[:, 4:7] == 0)                                                  # 1e: no input
    assert np.allclose(y[:, 7:12], x[:, 7:12] @ perm, atol=1e-14)


def test_linear_equivariance_and_backward():
    """Rotating every block by its Wigner matrix commutes with the mixing; the
    backward equals float64 autograd of the forward and a central difference."""
    from oracle import linear
    rng = np.random.default_rng(42)
    ins, outs = "4x0e+4x1o+4x2e+4x1o+4x3o", "5x0e+5x1o+5x2e+5x3o"
    jobs, d_in, d_out, c_in, c_out, nw = linear.plan(ins, outs)
    x = rng.standard_normal((6, d_in, c_in))
    W = rng.standard_normal(nw)
    R = wigner.random_rotation(rng)

    def rot(a, spec):
        a = a.copy()
        for (l, p, r, _) in linear.blocks(spec)[0]:
            D = wigner.wigner_d(l, R)
            a[:, r:r + 2 * l + 1] = np.einsum("ab,nbk->nak", D, a[:, r:r + 2 * l + 1])
        return a

    y = linear.forward(ins, outs, x, W).numpy()
    yr = linear.forward(ins, outs, rot(x, ins), W).numpy()
    assert np.allclose(yr, rot(y, outs), atol=1e-12)
    dout = rng.standard_normal((6, d_out, c_out))
    dx, dW = linear.backward(ins, outs, x, W, dout)
    xt = torch.tensor(x, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    L = (linear.forward(ins, outs, xt, Wt) * torch.as_tensor(dout)).sum()
    gx, gW = torch.autograd.grad(L, [xt, Wt])
    assert torch.allclose(dx, gx, atol=1e-12) and torch.allclose(dW, gW, atol=1e-12)
    u, v = rng.standard_normal(x.shape), rng.standard_normal(W.shape)
    f = lambda t: float((linear.forward(ins, outs, x + t * u, W + t * v) * torch.as_tensor(dout)).sum())
    h = 1e-3
    fd = (f(h) - f(-h)) / (2 * h)     # the loss is quadratic in t: exact up to rounding
    an = float((dx * torch.as_tensor(u)).sum() + (dW * torch.as_tensor(v)).sum())
    assert abs(fd - an) < 1e-8 * max(1.0, abs(an))


# ---------------------------------------------------------------- generic records
@pytest.mark.parametrize("spec", [("2x0e+2x1o+2x2e", 3, 3), ("3x0e+3x1o+3x2e+3x3o", 3, 3)])
def test_generic_records_equal_path_tp_and_backward(spec):
    """With the layout's own records and a shared y, the generic product equals
    the path-by-path product; with per-channel y equal to the shared one in every
    channel it equals it too; the backward equals float64 autograd of the forward
    (shared and per-channel y) and its dy sums over channels when y is shared."""
    from oracle import generic
    rng = np.random.default_rng(51)
    lay = irreps.layout(*spec)
    recs = cg.coo_records(lay)
    i0, i1, i2, v = (np.array([r[k] for r in recs]) for k in range(4))
    R, C = 5, lay.channels
    x = rng.standard_normal((R, lay.d_in, C))
    y = sh.sh_unit(lay.lmax_sh, _unit(rng, R))
    ref = tp.tp_unweighted(lay, x, y).numpy()
    assert np.allclose(generic.tp(i0, i1, i2, v, x, y, lay.d_out), ref, atol=1e-12)
    ypc = np.repeat(y[:, :, None], C, axis=2)
    assert np.allclose(generic.tp(i0, i1, i2, v, x, ypc, lay.d_out), ref, atol=1e-12)
    dz = rng.standard_normal(ref.shape)
    for yy in (y, ypc + rng.standard_normal(ypc.shape)):
        dx, dy = generic.tp_bwd(i0, i1, i2, v, x, yy, dz)
        xt = torch.tensor(x, requires_grad=True)
        yt = torch.tensor(yy, requires_grad=True)
        ye = yt if yy.ndim == 3 else yt[:, :, None]
        z = torch.zeros((R, lay.d_out, C), dtype=torch.float64)
        z = z.index_add(1, torch.as_tensor(i0), torch.as_tensor(v)[None, :, None] * xt[:, i1, :] * ye[:, i2, :])
        gx, gy = torch.autograd.grad((z * torch.as_tensor(dz)).sum(), [xt, yt])
        assert np.allclose(dx, gx.numpy(), atol=1e-11) and np.allclose(dy, gy.numpy(), atol=1e-11)


def test_generic_collapsed_output_block():
    """Records of two paths with the same output degree sent to one output block
    give the sum of the two paths' outputs (a collapsed output multiplicity)."""
    from oracle import generic
    rng = np.random.default_rng(52)
    lay = irreps.layout("2x0e+2x1o", 2, 1)
    recs = cg.coo_records(lay)
    blocks = [(p.out_off, p.l3) for p in lay.paths]
    # map every l3 = 1 block onto the first l3 = 1 block
    first1 = min(off for off, l3 in blocks if l3 == 1)
    remap = {}
    for off, l3 in blocks:
        for mm in range(2 * l3 + 1):
            remap[off + mm] = (first1 + mm) if l3 == 1 else off + mm
    i0 = np.array([remap[r[0]] for r in recs])
    i1, i2, v = (np.array([r[k] for r in recs]) for k in (1, 2, 3))
    x = rng.standard_normal((3, lay.d_in, lay.channels))
    y = sh.sh_unit(lay.lmax_sh, _unit(rng, 3))
    full = tp.tp_unweighted(lay, x, y).numpy()
    got = generic.tp(i0, i1, i2, v, x, y, lay.d_out)
    want = np.zeros_like(full)
    for off, l3 in blocks:
        if l3 == 1:
            want[:, first1:first1 + 3] += full[:, off:off + 3]
        else:
            want[:, off:off + 2 * l3 + 1] = full[:, off:off + 2 * l3 + 1]
    assert np.allclose(got, want, atol=1e-12)
