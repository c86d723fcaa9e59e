"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle.

Bar: relative L2 <= 1e-5 per floating-point output, bit-exact graph arrays,
bitwise-identical repeats.  Inputs are the seeded synthetic workloads; large
ones are checked on sampled rows the oracle computes one by one.
"""
import os

import numpy as np
import pytest

import synth
from oracle import conv as oconv
from oracle import graph as ograph
from oracle import irreps as oirreps
from oracle import radial as oradial
from oracle import sh as osh
from oracle import tp as otp

from gpu_util import (TOL, layout_of, oracle_bwd_rows, oracle_fwd_rows, rel_l2, to_dev, to_np,
                      upload_weights)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def e3():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2609_35099_amd import e3mi
    e3mi.lib()
    return e3mi


def _say(*a):
    print("[case]", *a, flush=True)


def _random_graph(rng, n, e, pad=-1):
    snd = rng.integers(0, n, e).astype(np.int32)
    rcv = rng.integers(0, n, e).astype(np.int32)
    rcv = np.where(rcv == snd, (rcv + 1) % n, rcv).astype(np.int32)
    vec = (rng.standard_normal((e, 3)) * 2.0).astype(np.float32)
    return snd, rcv, vec


# ---------------------------------------------------------------- graph
@pytest.mark.parametrize("case", ["cfg1", "random_pad", "empty", "isolated", "water8k", "three_passes",
                                  "four_passes", "whole_tiles", "two_nodes"])
def test_graph_csr_bit_exact(e3, case):
    """The CSR arrays equal the oracle's stable argsort bit for bit: one radix
    pass (N < 256), two (the 24,000-atom box), three (N = 300,000, with
    padding) and four (N above 2^24, edges on a few hundred nodes, so most keys
    repeat), edge counts that fill whole sort tiles, the smallest graphs."""
    _say("graph", case)
    rng = np.random.default_rng(1)
    pad = -1
    if case == "cfg1":
        g = synth.graph(synth.CONFIGS["cube64"])
        snd, rcv, n = g.sender, g.receiver, g.n_nodes
    elif case == "water8k":
        g = synth.graph(synth.CONFIGS["water8k"])
        snd, rcv, n = g.sender, g.receiver, g.n_nodes
    elif case == "random_pad":
        n = 300
        snd, rcv, _ = _random_graph(rng, n, 5000)
        pad = 17
    elif case == "three_passes":
        n = 300_000
        snd, rcv, _ = _random_graph(rng, n, 2_000_000)
        pad = 123_456
    elif case == "four_passes":
        n = (1 << 24) + 5
        hubs = rng.choice(n, 300, replace=False).astype(np.int32)
        snd = hubs[rng.integers(0, 300, 50_000)]
        rcv = hubs[rng.integers(0, 300, 50_000)]
    elif case == "whole_tiles":
        n = 700
        snd, rcv, _ = _random_graph(rng, n, 3 * 4096 + 1)
        snd, rcv = snd[:3 * 4096], rcv[:3 * 4096]
    elif case == "two_nodes":
        n = 2
        snd = np.array([0, 1, 1, 0, 1], np.int32)
        rcv = np.array([1, 0, 0, 1, 0], np.int32)
    elif case == "empty":
        n = 5
        snd = rcv = np.zeros(0, np.int32)
    else:
        n = 1000
        snd, rcv, _ = _random_graph(rng, 50, 700)   # nodes 50..999 isolated
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    pr, rr, ps, rs = (to_np(t) for t in G.export())
    ref = ograph.build(snd, rcv, n, pad)
    for got, want in zip((pr, rr, ps, rs), ref):
        assert np.array_equal(got.astype(np.int64), want)


def test_graph_rejects_out_of_range(e3):
    _say("graph out of range")
    snd = np.array([0, 1, 7], np.int32)
    rcv = np.array([1, 2, 0], np.int32)
    with pytest.raises(e3.E3Error) as ei:
        e3.Graph(to_dev(snd), to_dev(rcv), 5)
    assert ei.value.status == 3
    with pytest.raises(e3.E3Error):
        e3.Graph(to_dev(np.array([0, -1], np.int32)), to_dev(np.array([1, 1], np.int32)), 5)


# ---------------------------------------------------------------- harmonics
@pytest.mark.parametrize("lmax", [0, 1, 2, 3])
def test_sh_and_sh_bwd(e3, lmax):
    _say("sh", lmax)
    rng = np.random.default_rng(2)
    vec = (rng.standard_normal((1037, 3)) * 3).astype(np.float32)
    vec[5] = 0.0                                   # zero vector: Y_0 = 1, zeros, dvec = 0
    dy = rng.standard_normal((1037, (lmax + 1) ** 2)).astype(np.float32)
    y = to_np(e3.sh(lmax, to_dev(vec)))
    dv = to_np(e3.sh_bwd(lmax, to_dev(vec), to_dev(dy)))
    live = np.ones(1037, bool)
    live[5] = False
    ref_y = osh.sh_vec(lmax, vec[live].astype(np.float64))
    ref_dv = osh.sh_vec_vjp(lmax, vec[live].astype(np.float64), dy[live].astype(np.float64))
    assert rel_l2(y[live], ref_y) < TOL
    assert y[5, 0] == 1.0 and np.all(y[5, 1:] == 0.0)
    if lmax > 0:
        assert rel_l2(dv[live], ref_dv) < TOL
    assert np.all(dv[5] == 0.0)


# ---------------------------------------------------------------- tensor product
@pytest.mark.parametrize("irreps,lsh,lout,rows", [
    ("128x0e+128x1o+128x2e", 3, 3, 1001),   # the 200k-row layout, ragged batch tail
    ("64x0e+64x1o+64x2e", 3, 3, 77),
    ("8x0e+8x1o", 2, 2, 5),
    ("12x0e+12x1o+12x2e+12x3o", 3, 3, 33),    # C not a power of two
    ("100x0e+100x1o", 3, 3, 19),              # 50 lanes x 2 channels
    ("1024x0e+1024x1o+1024x2e", 3, 3, 9),     # the largest channel count
])
def test_tp_parity(e3, irreps, lsh, lout, rows):
    _say("tp", irreps, rows)
    plan = e3.Plan(irreps, lsh, lout)
    lay = oirreps.layout(irreps, lsh, lout)
    rng = np.random.default_rng(3)
    x = rng.standard_normal((rows, lay.d_in, lay.channels)).astype(np.float32)
    g = rng.standard_normal((rows, 3))
    y = osh.sh_unit(lsh, g / np.linalg.norm(g, axis=1, keepdims=True)).astype(np.float32)
    w = rng.standard_normal((rows, lay.n_paths, lay.channels)).astype(np.float32)
    z = to_np(e3.tp_fwd(plan, to_dev(x), to_dev(y), to_dev(w)))
    ref = otp.tp(lay, x, y, w).numpy()
    assert rel_l2(z, ref) < TOL
    z2 = to_np(e3.tp_fwd(plan, to_dev(x), to_dev(y), to_dev(w)))
    assert np.array_equal(z, z2)


def test_tp_200k_rows_full_size_sampled(e3):
    """The weighted TP at full size (200,000 rows, 128x0e+128x1o+128x2e, l <= 3),
    checked on sampled rows."""
    import torch
    _say("tp 200k rows full")
    cfg = synth.CONFIGS["tp200k"]
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    lay = layout_of(cfg)
    x, u, w = synth.tp_inputs(cfg)
    y = osh.sh_unit(3, u.astype(np.float64)).astype(np.float32)
    z = e3.tp_fwd(plan, to_dev(x), to_dev(y), to_dev(w))
    torch.cuda.synchronize()
    rows = np.concatenate([[0, 1, 7, 8, 199_999], np.random.default_rng(4).integers(0, 200_000, 59)])
    got = to_np(z[torch.as_tensor(rows, device="cuda")])
    ref = otp.tp(lay, x[rows], y[rows], w[rows]).numpy()
    assert rel_l2(got, ref) < TOL


@pytest.mark.parametrize("irreps,lsh,lout,rows", [
    ("128x0e+128x1o+128x2e", 3, 3, 1001),
    ("64x0e+64x1o+64x2e", 3, 3, 77),
    ("8x0e+8x1o", 2, 2, 5),
    ("12x0e+12x1o+12x2e+12x3o", 3, 3, 33),
    ("100x0e+100x1o", 3, 3, 19),
    ("4x0e+4x1o", 3, 3, 1),
    ("1024x0e+1024x1o+1024x2e", 3, 3, 5),
])
def test_tp_bwd_parity(e3, irreps, lsh, lout, rows):
    _say("tp bwd", irreps, rows)
    plan = e3.Plan(irreps, lsh, lout)
    lay = oirreps.layout(irreps, lsh, lout)
    rng = np.random.default_rng(5)
    x = rng.standard_normal((rows, lay.d_in, lay.channels)).astype(np.float32)
    g = rng.standard_normal((rows, 3))
    y = osh.sh_unit(lsh, g / np.linalg.norm(g, axis=1, keepdims=True)).astype(np.float32)
    w = rng.standard_normal((rows, lay.n_paths, lay.channels)).astype(np.float32)
    dz = rng.standard_normal((rows, lay.d_out, lay.channels)).astype(np.float32)
    args = [to_dev(a) for a in (x, y, w, dz)]
    dx, dy, dw = (to_np(t) for t in e3.tp_bwd(plan, *args))
    rdx, rdy, rdw = (t.numpy() for t in otp.tp_bwd(lay, x, y, w, dz))
    errs = dict(dx=rel_l2(dx, rdx), dy=rel_l2(dy, rdy), dw=rel_l2(dw, rdw))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    again = [to_np(t) for t in e3.tp_bwd(plan, *args)]
    for u, v in zip((dx, dy, dw), again):
        assert np.array_equal(u, v)


def test_tp_bwd_200k_rows_full_size_sampled(e3):
    """TP backward at full size (200,000 rows), checked on sampled rows."""
    import torch
    _say("tp bwd 200k rows full")
    cfg = synth.CONFIGS["tp200k"]
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    lay = layout_of(cfg)
    x, u, w = synth.tp_inputs(cfg)
    y = osh.sh_unit(3, u.astype(np.float64)).astype(np.float32)
    R = x.shape[0]
    dz = synth.normal_device(cfg.cid, synth._DM, (R, lay.d_out, lay.channels), "cuda")
    dx, dy, dw = e3.tp_bwd(plan, to_dev(x), to_dev(y), to_dev(w), dz)
    torch.cuda.synchronize()
    rows = np.concatenate([[0, 1, 7, 8, R - 1], np.random.default_rng(6).integers(0, R, 59)])
    ri = torch.as_tensor(rows, device="cuda")
    ref = otp.tp_bwd(lay, x[rows], y[rows], w[rows], to_np(dz[ri]))
    for name, got, r in zip(("dx", "dy", "dw"), (dx, dy, dw), ref):
        err = rel_l2(to_np(got[ri]), r.numpy())
        print(name, err, flush=True)
        assert err < TOL, (name, err)


# ---------------------------------------------------------------- convolution
def _run_conv(e3, plan, snd, rcv, n, vec, x, s, dm, pad=-1):
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    xs, vs, ss, ds_ = to_dev(x), to_dev(vec), to_dev(s), to_dev(dm)
    m = e3.conv_fwd(plan, G, xs, vs, ss)
    dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, ss, ds_)
    return G, m, dx, dvec, ds


def _check_full(lay, snd, rcv, n, vec, x, s, dm, m, dx, dvec, ds, pad=-1):
    ref_m = oconv.conv_fwd(lay, x, vec, s, snd, rcv, n, pad_node=pad).numpy()
    ref = oconv.conv_bwd(lay, x, vec, s, dm, snd, rcv, n, pad_node=pad)
    errs = dict(m=rel_l2(to_np(m), ref_m), dx=rel_l2(to_np(dx), ref["dx"].numpy()),
                ds=rel_l2(to_np(ds), ref["ds"].numpy()), dvec=rel_l2(to_np(dvec), ref["dvec"].numpy()))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    return ref_m, ref


def test_conv_cube64_full(e3):
    """64 atoms in a cube, 8x0e+8x1o, harmonics and outputs to l = 2: full oracle."""
    _say("conv cube64")
    cfg = synth.CONFIGS["cube64"]
    g = synth.graph(cfg)
    x = synth.node_features(cfg, g.n_nodes)
    s = synth.edge_weights(cfg, g.vec, 0, g.sender.shape[0])
    dm = synth.out_cotangent(cfg, g.n_nodes)
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    G, m, dx, dvec, ds = _run_conv(e3, plan, g.sender, g.receiver, g.n_nodes, g.vec, x, s, dm)
    _check_full(layout_of(cfg), g.sender, g.receiver, g.n_nodes, g.vec, x, s, dm, m, dx, dvec, ds)


@pytest.mark.parametrize("irreps,lsh,lout,n,e,pad", [
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, 120, 2500, -1),
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, 90, 1800, 7),
    ("64x0e+64x1o+64x2e+64x3o", 3, 3, 70, 1500, -1),
    ("128x0e+128x1o", 3, 3, 200, 4000, -1),
    ("16x0e+16x1o+16x2e", 3, 3, 40, 600, 3),
    ("128x0e+128x1o+128x2e", 3, 3, 50, 900, -1),
    ("32x0e+32x1o+32x2e", 2, 2, 60, 900, -1),          # l_max 2 variant
    ("256x0e+256x1o+256x2e", 2, 2, 30, 300, 4),
    ("1024x0e+1024x1o+1024x2e+1024x3o", 3, 3, 12, 60, -1),   # the largest channel count
])
def test_conv_random_graphs_full(e3, irreps, lsh, lout, n, e, pad):
    _say("conv random", irreps, n, e, pad)
    rng = np.random.default_rng(5)
    lay = oirreps.layout(irreps, lsh, lout)
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
    s = rng.standard_normal((e, lay.n_paths, C)).astype(np.float32)
    dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
    plan = e3.Plan(irreps, lsh, lout)
    G, m, dx, dvec, ds = _run_conv(e3, plan, snd, rcv, n, vec, x, s, dm, pad)
    _check_full(lay, snd, rcv, n, vec, x, s, dm, m, dx, dvec, ds, pad)
    if pad >= 0:
        dead = (snd == pad) | (rcv == pad)
        assert np.all(to_np(ds)[dead] == 0) and np.all(to_np(dvec)[dead] == 0)
        assert np.all(to_np(m)[pad] == 0) and np.all(to_np(dx)[pad] == 0)


@pytest.mark.parametrize("irreps,lsh,lout,parity,n,e,pad", [
    ("8x0e+8x1o", 2, 2, "natural", 64, 900, -1),                         # the 64-atom cube's blocks
    ("128x0e+128x1o", 3, 3, "natural", 120, 2500, 9),
    ("32x0e+32x1o+32x2e", 3, 3, "natural", 80, 1300, -1),
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, "natural", 90, 1800, 7),      # the benchmark's blocks
    ("128x0o+128x1e+128x2o+128x3e", 3, 3, "all", 60, 1100, -1),         # other parities, same kernels
    ("128x1o+128x0e+128x3o+128x2e", 3, 3, "all", 100, 2100, 4),         # blocks out of degree order
])
def test_layout_variants_conv_and_tp(e3, irreps, lsh, lout, parity, n, e, pad):
    """Natural-parity path sets and a reordered block list: convolution forward
    and backward and the tensor product forward and backward, against the
    oracle's layout of the same parity reading."""
    _say("layout variant", irreps, parity, n, e, pad)
    rng = np.random.default_rng(15)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = e3.Plan(irreps, lsh, lout, natural=parity == "natural")
    assert plan.supported and (plan.P, plan.D_out) == (lay.n_paths, lay.d_out)
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
    s = rng.standard_normal((e, lay.n_paths, C)).astype(np.float32)
    dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
    G, m, dx, dvec, ds = _run_conv(e3, plan, snd, rcv, n, vec, x, s, dm, pad)
    _check_full(lay, snd, rcv, n, vec, x, s, dm, m, dx, dvec, ds, pad)
    rows = 37
    g = rng.standard_normal((rows, 3))
    y = osh.sh_unit(lsh, g / np.linalg.norm(g, axis=1, keepdims=True)).astype(np.float32)
    xt = rng.standard_normal((rows, lay.d_in, C)).astype(np.float32)
    w = rng.standard_normal((rows, lay.n_paths, C)).astype(np.float32)
    dz = rng.standard_normal((rows, lay.d_out, C)).astype(np.float32)
    z = to_np(e3.tp_fwd(plan, to_dev(xt), to_dev(y), to_dev(w)))
    assert rel_l2(z, otp.tp(lay, xt, y, w).numpy()) < TOL
    got = [to_np(t) for t in e3.tp_bwd(plan, to_dev(xt), to_dev(y), to_dev(w), to_dev(dz))]
    for a, r in zip(got, otp.tp_bwd(lay, xt, y, w, dz)):
        assert rel_l2(a, r.numpy()) < TOL


def test_conv_degenerate_graphs(e3):
    """No edges; a single edge; nodes without in-edges."""
    irreps = "128x0e+128x1o+128x2e+128x3o"
    lay = oirreps.layout(irreps, 3, 3)
    plan = e3.Plan(irreps, 3, 3)
    rng = np.random.default_rng(6)
    for snd, rcv, n in [(np.zeros(0, np.int32), np.zeros(0, np.int32), 4),
                        (np.array([2], np.int32), np.array([0], np.int32), 3)]:
        _say("conv degenerate", len(snd))
        e = len(snd)
        vec = rng.standard_normal((e, 3)).astype(np.float32)
        x = rng.standard_normal((n, lay.d_in, 128)).astype(np.float32)
        s = rng.standard_normal((e, lay.n_paths, 128)).astype(np.float32)
        dm = rng.standard_normal((n, lay.d_out, 128)).astype(np.float32)
        G, m, dx, dvec, ds = _run_conv(e3, plan, snd, rcv, n, vec, x, s, dm)
        if e == 0:
            assert np.all(to_np(m) == 0) and np.all(to_np(dx) == 0)
        else:
            _check_full(lay, snd, rcv, n, vec, x, s, dm, m, dx, dvec, ds)
            assert np.all(to_np(m)[1:] == 0)


def test_conv_deterministic_and_invariants(e3):
    """Bitwise-identical repeats; trilinear identity and dvec . r = 0 on GPU outputs."""
    import torch
    _say("conv determinism water1k")
    cfg = synth.CONFIGS["water1k"]
    g = synth.graph(cfg)
    x = synth.node_features(cfg, g.n_nodes)
    dm = synth.out_cotangent(cfg, g.n_nodes)
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    s = upload_weights(cfg, g.vec)
    G = e3.Graph(to_dev(g.sender), to_dev(g.receiver), g.n_nodes)
    xs, vs, dms = to_dev(x), to_dev(g.vec), to_dev(dm)
    outs = []
    for _ in range(3):
        m = e3.conv_fwd(plan, G, xs, vs, s)
        dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, s, dms)
        outs.append((m.clone(), dx.clone(), dvec.clone(), ds.clone()))
    torch.cuda.synchronize()
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert torch.equal(a, b)
    m, dx, dvec, ds = outs[0]
    ym = e3.sh(3, vs)
    t_m = float((m.double() * dms.double()).sum())
    t_x = float((dx.double() * xs.double()).sum())
    t_s = float((ds.double() * s.double()).sum())
    assert abs(t_x - t_m) < 1e-5 * abs(t_m) and abs(t_s - t_m) < 1e-5 * abs(t_m)
    radial = (dvec.double() * vs.double()).sum(1).abs()
    scale = dvec.double().norm(dim=1) * vs.double().norm(dim=1)
    assert float((radial / scale.clamp_min(1e-30)).max()) < 1e-4
    # sampled oracle rows
    lay = layout_of(cfg)
    rng = np.random.default_rng(7)
    rs = rng.choice(g.n_nodes, 40, replace=False)
    es = rng.choice(g.sender.shape[0], 100, replace=False)
    W = synth.bessel_matrix(cfg)
    sfn = lambda rows: synth.edge_weights_rows(cfg, g.vec, rows, W=W)
    ref_m = oracle_fwd_rows(lay, x, g.vec, sfn, g.sender, g.receiver, g.n_nodes, rs)
    ref_dx, ref_ds, ref_dv = oracle_bwd_rows(lay, x, g.vec, sfn, dm, g.sender, g.receiver, g.n_nodes, rs, es)
    assert rel_l2(to_np(m)[rs], ref_m) < TOL
    assert rel_l2(to_np(dx)[rs], ref_dx) < TOL
    assert rel_l2(to_np(ds)[es], ref_ds) < TOL
    assert rel_l2(to_np(dvec)[es], ref_dv) < TOL


@pytest.mark.parametrize("name", ["water8k"])
def test_conv_full_size_sampled(e3, name):
    """The benchmark workload (24,000-atom water box, l<=3, 128 channels) at full
    size, in the launch configuration the benchmark times, on sampled rows."""
    import torch
    _say("conv full size", name)
    cfg = synth.CONFIGS[name]
    g = synth.graph(cfg)
    x = synth.node_features(cfg, g.n_nodes)
    dm = synth.out_cotangent(cfg, g.n_nodes)
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    s = upload_weights(cfg, g.vec)
    G = e3.Graph(to_dev(g.sender), to_dev(g.receiver), g.n_nodes)
    xs, vs, dms = to_dev(x), to_dev(g.vec), to_dev(dm)
    m = e3.conv_fwd(plan, G, xs, vs, s)
    dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, s, dms)
    torch.cuda.synchronize()
    lay = layout_of(cfg)
    rng = np.random.default_rng(8)
    E = g.sender.shape[0]
    rs = np.concatenate([[0, g.n_nodes - 1], rng.choice(g.n_nodes, 22, replace=False)])
    es = np.concatenate([[0, E - 1], rng.choice(E, 62, replace=False)])
    W = synth.bessel_matrix(cfg) if cfg.weights == "bessel" else None
    sfn = lambda rows: synth.edge_weights_rows(cfg, g.vec, rows, W=W)
    ref_m = oracle_fwd_rows(lay, x, g.vec, sfn, g.sender, g.receiver, g.n_nodes, rs)
    ref_dx, ref_ds, ref_dv = oracle_bwd_rows(lay, x, g.vec, sfn, dm, g.sender, g.receiver, g.n_nodes, rs, es)
    ri = torch.as_tensor(rs, device="cuda")
    ei = torch.as_tensor(es, device="cuda")
    errs = dict(m=rel_l2(to_np(m[ri]), ref_m), dx=rel_l2(to_np(dx[ri]), ref_dx),
                ds=rel_l2(to_np(ds[ei]), ref_ds), dvec=rel_l2(to_np(dvec[ei]), ref_dv))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)


# ---------------------------------------------------------------- fused radial weights
def _radial_full(e3, plan, lay, snd, rcv, n, vec, x, h, W, dm, pad=-1, repeat=2):
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    xs, vs, hs, Ws, dms = (to_dev(a) for a in (x, vec, h, W, dm))
    outs = []
    for _ in range(repeat):
        m = e3.conv_fwd_radial(plan, G, xs, vs, hs, Ws)
        outs.append((m,) + e3.conv_bwd_radial(plan, G, xs, vs, hs, Ws, dms))
    outs = [[to_np(t) for t in o] for o in outs]
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert np.array_equal(a, b), "not deterministic"
    m, dx, dvec, dh, dW = outs[0]
    ref_m = oradial.conv_fwd(lay, x, vec, h, W, snd, rcv, n, pad_node=pad).numpy()
    ref = oradial.conv_bwd(lay, x, vec, h, W, dm, snd, rcv, n, pad_node=pad)
    errs = dict(m=rel_l2(m, ref_m), dx=rel_l2(dx, ref["dx"].numpy()), dvec=rel_l2(dvec, ref["dvec"].numpy()),
                dh=rel_l2(dh, ref["dh"].numpy()), dW=rel_l2(dW, ref["dW"].numpy()))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    return m, dx, dvec, dh, dW


@pytest.mark.parametrize("irreps,lsh,lout,n,e,K,pad", [
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, 100, 2000, 8, -1),
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, 60, 1200, 16, 5),
    ("64x0e+64x1o+64x2e+64x3o", 3, 3, 50, 900, 5, -1),
    ("16x0e+16x1o+16x2e", 3, 3, 40, 600, 1, 3),
    ("8x0e+8x1o", 2, 2, 30, 300, 12, -1),
    ("100x0e+100x1o", 3, 3, 40, 700, 8, -1),   # 64 + 36 channel lanes
])
def test_conv_radial_random_graphs_full(e3, irreps, lsh, lout, n, e, K, pad):
    _say("conv radial", irreps, n, e, K, pad)
    rng = np.random.default_rng(11)
    lay = oirreps.layout(irreps, lsh, lout)
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
    h = rng.standard_normal((e, K)).astype(np.float32)
    W = (rng.standard_normal((K, lay.n_paths, C)) / np.sqrt(K)).astype(np.float32)
    dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
    plan = e3.Plan(irreps, lsh, lout)
    m, dx, dvec, dh, dW = _radial_full(e3, plan, lay, snd, rcv, n, vec, x, h, W, dm, pad)
    if pad >= 0:
        dead = (snd == pad) | (rcv == pad)
        assert np.all(dh[dead] == 0) and np.all(dvec[dead] == 0)
        assert np.all(m[pad] == 0) and np.all(dx[pad] == 0)


def test_conv_radial_degenerate_graphs(e3):
    """No edges (dW = 0, m = 0); a single edge."""
    irreps = "128x0e+128x1o+128x2e+128x3o"
    lay = oirreps.layout(irreps, 3, 3)
    plan = e3.Plan(irreps, 3, 3)
    rng = np.random.default_rng(12)
    K = 8
    W = rng.standard_normal((K, lay.n_paths, 128)).astype(np.float32)
    for snd, rcv, n in [(np.zeros(0, np.int32), np.zeros(0, np.int32), 4),
                        (np.array([2], np.int32), np.array([0], np.int32), 3)]:
        _say("conv radial degenerate", len(snd))
        e = len(snd)
        vec = rng.standard_normal((e, 3)).astype(np.float32)
        x = rng.standard_normal((n, lay.d_in, 128)).astype(np.float32)
        h = rng.standard_normal((e, K)).astype(np.float32)
        dm = rng.standard_normal((n, lay.d_out, 128)).astype(np.float32)
        if e == 0:
            G = e3.Graph(to_dev(snd), to_dev(rcv), n)
            xs, Ws = to_dev(x), to_dev(W)
            vs = to_dev(vec.reshape(0, 3))
            hs = to_dev(h.reshape(0, K))
            m = e3.conv_fwd_radial(plan, G, xs, vs, hs, Ws)
            dx, dvec, dh, dW = e3.conv_bwd_radial(plan, G, xs, vs, hs, Ws, to_dev(dm))
            assert np.all(to_np(m) == 0) and np.all(to_np(dx) == 0) and np.all(to_np(dW) == 0)
        else:
            m = _radial_full(e3, plan, lay, snd, rcv, n, vec, x, h, W, dm, repeat=1)[0]
            assert np.all(m[1:] == 0)


def test_conv_radial_water8k_sampled(e3):
    """The 24,000-atom water box with its own radial recipe fused: h = the
    8-function Bessel basis of |r|, W = the workload's fixed matrix.  m, dx, dvec
    and dh are checked against the oracle on sampled rows.  dW sums over all
    1.27M edges, which the oracle cannot do in seconds: it is checked against a
    float64 sum of h_e ds_e with ds from the plain backward (itself checked
    against the oracle in test_conv_full_size_sampled)."""
    import torch
    _say("conv radial water8k full")
    cfg = synth.CONFIGS["water8k"]
    g = synth.graph(cfg)
    x = synth.node_features(cfg, g.n_nodes)
    dm = synth.out_cotangent(cfg, g.n_nodes)
    h, W = synth.radial_inputs(cfg, g.vec)
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    G = e3.Graph(to_dev(g.sender), to_dev(g.receiver), g.n_nodes)
    xs, vs, hs, Ws, dms = (to_dev(a) for a in (x, g.vec, h, W, dm))
    m = e3.conv_fwd_radial(plan, G, xs, vs, hs, Ws)
    dx, dvec, dh, dW = e3.conv_bwd_radial(plan, G, xs, vs, hs, Ws, dms)
    torch.cuda.synchronize()
    lay = layout_of(cfg)
    rng = np.random.default_rng(13)
    E = g.sender.shape[0]
    rs = np.concatenate([[0, g.n_nodes - 1], rng.choice(g.n_nodes, 22, replace=False)])
    es = np.concatenate([[0, E - 1], rng.choice(E, 62, replace=False)])
    sfn = lambda rows: oradial.weights(h[rows], W).numpy()
    ref_m = oracle_fwd_rows(lay, x, g.vec, sfn, g.sender, g.receiver, g.n_nodes, rs)
    ref_dx, ref_ds, ref_dv = oracle_bwd_rows(lay, x, g.vec, sfn, dm, g.sender, g.receiver, g.n_nodes, rs, es)
    ref_dh = np.einsum("ekq,jkq->ej", ref_ds, W.astype(np.float64))
    ri, ei = torch.as_tensor(rs, device="cuda"), torch.as_tensor(es, device="cuda")
    errs = dict(m=rel_l2(to_np(m[ri]), ref_m), dx=rel_l2(to_np(dx[ri]), ref_dx),
                dvec=rel_l2(to_np(dvec[ei]), ref_dv), dh=rel_l2(to_np(dh[ei]), ref_dh))
    del m
    # dW against a float64 sum over the plain backward's ds
    s = torch.empty((E, plan.P, plan.C), dtype=torch.float32, device="cuda")
    W64 = Ws.double().reshape(W.shape[0], -1)
    for e0 in range(0, E, 1 << 16):
        e1 = min(E, e0 + (1 << 16))
        s[e0:e1] = (hs[e0:e1].double() @ W64).float().reshape(e1 - e0, plan.P, plan.C)
    ds = e3.conv_bwd(plan, G, xs, vs, s, dms)[2]
    del s
    acc = torch.zeros_like(W64)
    for e0 in range(0, E, 1 << 16):
        e1 = min(E, e0 + (1 << 16))
        acc += hs[e0:e1].double().T @ ds[e0:e1].double().reshape(e1 - e0, -1)
    errs["dW"] = rel_l2(to_np(dW).reshape(acc.shape), acc.cpu().numpy())
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)


# ---------------------------------------------------------------- harmonics as input; double backward
@pytest.mark.parametrize("irreps,lsh,lout,n,e,pad", [
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, 80, 1500, -1),
    ("64x0e+64x1o+64x2e", 3, 3, 50, 800, 4),
    ("8x0e+8x1o", 2, 2, 20, 150, -1),
])
def test_conv_y_input_accumulate_and_optional_outputs(e3, irreps, lsh, lout, n, e, pad):
    """conv and conv_bwd with an arbitrary y (not harmonics) against the oracle;
    accumulate adds; an omitted cotangent leaves the others unchanged."""
    import torch
    _say("conv y-input", irreps, n, e, pad)
    rng = np.random.default_rng(14)
    lay = oirreps.layout(irreps, lsh, lout)
    snd, rcv, _ = _random_graph(rng, n, e)
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
    y = rng.standard_normal((e, lay.d_sh)).astype(np.float32)
    s = rng.standard_normal((e, lay.n_paths, C)).astype(np.float32)
    dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
    plan = e3.Plan(irreps, lsh, lout)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    xs, ys, ss, dms = (to_dev(a) for a in (x, y, s, dm))
    m = e3.conv_fwd_y(plan, G, xs, ys, ss)
    dx, dy, ds = e3.conv_bwd_y(plan, G, xs, ys, ss, dms)
    ref_m = oconv.conv_fwd_from_y(lay, x, y, s, snd, rcv, n, pad_node=pad).numpy()
    ref = oconv.conv_bwd_from_y(lay, x, y, s, dm, snd, rcv, n, pad_node=pad)
    errs = dict(m=rel_l2(to_np(m), ref_m), dx=rel_l2(to_np(dx), ref["dx"].numpy()),
                dy=rel_l2(to_np(dy), ref["dy"].numpy()), ds=rel_l2(to_np(ds), ref["ds"].numpy()))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    # accumulate: a second call adds the same values (x + x is exact in binary)
    m2 = m.clone()
    e3.conv_fwd_y(plan, G, xs, ys, ss, out=m2, accumulate=True)
    d2 = [t.clone() for t in (dx, dy, ds)]
    e3.conv_bwd_y(plan, G, xs, ys, ss, dms, dx=d2[0], dy=d2[1], ds=d2[2], accumulate=True)
    assert torch.equal(m2, 2 * m)
    for a, b in zip(d2, (dx, dy, ds)):
        assert torch.equal(a, 2 * b)
    # omitted cotangents: the stored ones are bit-identical
    for want in (("dx",), ("dy",), ("ds",), ("dy", "ds")):
        got = e3.conv_bwd_y(plan, G, xs, ys, ss, dms, want=want)
        for name, full, part in zip(("dx", "dy", "ds"), (dx, dy, ds), got):
            if name in want:
                assert torch.equal(full, part), (want, name)
            else:
                assert part is None


@pytest.mark.parametrize("irreps,lsh,lout,n,e,pad", [
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, 60, 1000, -1),
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, 40, 700, 6),
    ("16x0e+16x1o+16x2e", 3, 3, 30, 400, -1),
    ("8x0e+8x1o", 2, 2, 20, 150, 2),
    ("132x0e+132x1o", 2, 2, 25, 300, -1),  # three channel slabs, the last of four channels
])
def test_conv_bwd2_random_graphs_full(e3, irreps, lsh, lout, n, e, pad):
    import torch
    _say("conv bwd2", irreps, n, e, pad)
    rng = np.random.default_rng(15)
    lay = oirreps.layout(irreps, lsh, lout)
    snd, rcv, _ = _random_graph(rng, n, e)
    C = lay.channels
    arrs = dict(x=(n, lay.d_in, C), y=(e, lay.d_sh), s=(e, lay.n_paths, C), dm=(n, lay.d_out, C),
                ddx=(n, lay.d_in, C), ddy=(e, lay.d_sh), dds=(e, lay.n_paths, C))
    a = {k: rng.standard_normal(v).astype(np.float32) for k, v in arrs.items()}
    plan = e3.Plan(irreps, lsh, lout)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    d = {k: to_dev(v) for k, v in a.items()}
    outs = [e3.conv_bwd2(plan, G, d["x"], d["y"], d["s"], d["dm"], d["ddx"], d["ddy"], d["dds"]) for _ in range(2)]
    for u, v in zip(*outs):
        assert torch.equal(u, v)
    ref = oconv.conv_bwd2(lay, a["x"], a["y"], a["s"], a["dm"], a["ddx"], a["ddy"], a["dds"], snd, rcv, n,
                          pad_node=pad)
    errs = {k: rel_l2(to_np(g), ref[k].numpy()) for k, g in zip(("dx", "dy", "ds", "ddm"), outs[0])}
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    if pad >= 0:
        dead = (snd == pad) | (rcv == pad)
        assert np.all(to_np(outs[0][1])[dead] == 0) and np.all(to_np(outs[0][2])[dead] == 0)


def test_conv_bwd2_water8k_sampled(e3):
    """Double backward on the 24,000-atom water box (y its harmonics) at full
    size; checked on a compact sub-problem holding every in-edge of the sampled
    receivers, every out-edge of the sampled senders and the sampled edges."""
    import torch
    _say("conv bwd2 water8k full")
    cfg = synth.CONFIGS["water8k"]
    g = synth.graph(cfg)
    N, E = g.n_nodes, g.sender.shape[0]
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    lay = layout_of(cfg)
    dev = torch.device("cuda")
    x = synth.node_features(cfg, N)
    dm = synth.out_cotangent(cfg, N)
    rng = np.random.default_rng(16)
    ddx = rng.standard_normal(x.shape).astype(np.float32)
    G = e3.Graph(to_dev(g.sender), to_dev(g.receiver), N)
    vs = to_dev(g.vec)
    ys = e3.sh(cfg.lmax_sh, vs)
    ddy = torch.randn((E, plan.D_sh), device=dev, generator=torch.Generator(device=dev).manual_seed(17))
    s = upload_weights(cfg, g.vec)
    dds = synth.normal_device(cfg.cid, 9, (E, plan.P, plan.C), dev)
    xs, dms, ddxs = to_dev(x), to_dev(dm), to_dev(ddx)
    gx, gy, gs, gdm = e3.conv_bwd2(plan, G, xs, ys, s, dms, ddxs, ddy, dds)
    torch.cuda.synchronize()
    rs = np.concatenate([[0, N - 1], rng.choice(N, 10, replace=False)])
    es = np.concatenate([[0, E - 1], rng.choice(E, 30, replace=False)])
    sel = np.unique(np.concatenate([np.nonzero(np.isin(g.receiver, rs))[0],
                                    np.nonzero(np.isin(g.sender, rs))[0], es]))
    nodes, inv = np.unique(np.concatenate([g.sender[sel], g.receiver[sel]]), return_inverse=True)
    sc, rc = inv[:sel.shape[0]], inv[sel.shape[0]:]
    ed = torch.as_tensor(sel, device=dev)
    take = lambda t: t[ed].cpu().numpy()
    ref = oconv.conv_bwd2(lay, x[nodes], take(ys), take(s), dm[nodes], ddx[nodes], take(ddy), take(dds),
                          sc, rc, nodes.shape[0])
    ni = np.searchsorted(nodes, rs)
    ep = np.searchsorted(sel, es)
    ri, ei = torch.as_tensor(rs, device=dev), torch.as_tensor(es, device=dev)
    errs = dict(dx=rel_l2(to_np(gx[ri]), ref["dx"].numpy()[ni]), ddm=rel_l2(to_np(gdm[ri]), ref["ddm"].numpy()[ni]),
                dy=rel_l2(to_np(gy[ei]), ref["dy"].numpy()[ep]), ds=rel_l2(to_np(gs[ei]), ref["ds"].numpy()[ep]))
    print("rel-L2", errs, f"(sub-problem: {sel.shape[0]} edges, {nodes.shape[0]} nodes)", flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)


# ---------------------------------------------------------------- linear mixing
from oracle import linear as olinear  # noqa: E402


@pytest.mark.parametrize("ins,outs,n", [
    ("16x0e+16x1o+16x1o+16x2e", "32x0e+32x1o+32x1e+32x2e", 37),      # two 1o inputs; 1e has none
    ("128x0e+128x1o+128x2e+128x3o", "128x0e+128x1o+128x2e+128x3o", 101),
    ("64x0e+64x1o", "192x0e+192x1o", 9),                              # 3 column slabs
    ("48x1o+48x0e+48x1o+48x1o", "16x1o+16x0e", 23),
    ("512x0e+512x1o", "1024x0e+1024x1o", 13),                       # large multiplicities
])
def test_linear_small_full(e3, ins, outs, n):
    import torch
    _say("linear", ins, "->", outs, n)
    L = e3.Linear(ins, outs)
    rng = np.random.default_rng(18)
    x = rng.standard_normal((n, L.D_in, L.C_in)).astype(np.float32)
    W = (rng.standard_normal(L.n_weights) / 8).astype(np.float32)
    dout = rng.standard_normal((n, L.D_out, L.C_out)).astype(np.float32)
    xs, Ws, ds = to_dev(x), to_dev(W), to_dev(dout)
    y = L.forward(xs, Ws)
    dx, dW = L.backward(xs, Ws, ds)
    y2 = L.forward(xs, Ws)
    dx2, dW2 = L.backward(xs, Ws, ds)
    assert torch.equal(y, y2) and torch.equal(dx, dx2) and torch.equal(dW, dW2)
    ref_y = olinear.forward(ins, outs, x, W).numpy()
    ref_dx, ref_dW = (t.numpy() for t in olinear.backward(ins, outs, x, W, dout))
    errs = dict(y=rel_l2(to_np(y), ref_y), dx=rel_l2(to_np(dx), ref_dx), dW=rel_l2(to_np(dW), ref_dW))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)


def _path_irreps(plan):
    """Irreps string of the convolution's output blocks (one block per path)."""
    names = []
    for l1, l2, l3, p3, x_off, y_off, out_off in plan.paths():
        names.append(f"{plan.C}x{l3}{'e' if p3 > 0 else 'o'}")
    return "+".join(names)


@pytest.mark.parametrize("which", ["nodes", "messages"])
def test_linear_water8k_sampled(e3, which):
    """Full-size mixing on 24,000 nodes, 128 channels: node features
    (x blocks 0e,1o,2e,3o), or the convolution output (34 path blocks mixed per
    degree and parity).  Outputs on sampled nodes; dW on sampled pairs, each from
    an oracle sub-problem holding only that pair's two blocks over all nodes."""
    import torch
    cfg = synth.CONFIGS["water8k"]
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    N = 24000
    ins = cfg.irreps if which == "nodes" else _path_irreps(plan)
    outs = "128x0e+128x1o+128x2e+128x3o" if which == "nodes" else \
        "128x0e+128x0o+128x1o+128x1e+128x2e+128x2o+128x3o+128x3e"
    _say("linear water8k", which, ins[:40], "->", outs)
    L = e3.Linear(ins, outs)
    dev = torch.device("cuda")
    xs = synth.normal_device(4, 20, (N, L.D_in, L.C_in), dev)
    Ws = synth.normal_device(4, 21, (L.n_weights,), dev) / 16
    ds = synth.normal_device(4, 22, (N, L.D_out, L.C_out), dev)
    y = L.forward(xs, Ws)
    dx, dW = L.backward(xs, Ws, ds)
    torch.cuda.synchronize()
    rng = np.random.default_rng(19)
    rows = np.concatenate([[0, N - 1], rng.choice(N, 30, replace=False)])
    ri = torch.as_tensor(rows, device=dev)
    x_r, d_r, W_h = to_np(xs[ri]), to_np(ds[ri]), to_np(Ws)
    errs = dict(y=rel_l2(to_np(y[ri]), olinear.forward(ins, outs, x_r, W_h).numpy()),
                dx=rel_l2(to_np(dx[ri]), olinear.backward(ins, outs, x_r, W_h, d_r)[0].numpy()))
    jobs = olinear.plan(ins, outs)[0]
    bi = olinear.blocks(ins)[0]
    bo = olinear.blocks(outs)[0]
    pairs = [(o, t) for o, job in enumerate(jobs) for t in range(len(job[2]))]
    for o, t in [pairs[i] for i in rng.choice(len(pairs), 3, replace=False)]:
        l, orow, src, off, n = jobs[o]
        irow = src[t]
        R = 2 * l + 1
        sub_in = f"{L.C_in}x{l}{'e' if bo[o][1] > 0 else 'o'}"
        sub_out = f"{L.C_out}x{l}{'e' if bo[o][1] > 0 else 'o'}"
        xb = to_np(xs[:, irow:irow + R])
        db = to_np(ds[:, orow:orow + R])
        ref = olinear.backward(sub_in, sub_out, xb, np.zeros(L.C_in * L.C_out), db)[1].numpy()
        got = to_np(dW[off + t * L.C_in * L.C_out: off + (t + 1) * L.C_in * L.C_out])
        errs[f"dW[{o},{t}]"] = rel_l2(got, ref)
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)


# ---------------------------------------------------------------- caller-supplied records
from oracle import cg as ocg  # noqa: E402
from oracle import generic as ogeneric  # noqa: E402


def _layout_records(lay):
    recs = ocg.coo_records(lay)
    return tuple(np.array([r[k] for r in recs]) for k in range(4))


@pytest.mark.parametrize("case", ["layout-shared", "layout-perchannel", "random-shared", "random-perchannel",
                                  "collapsed", "C7", "layout-l2in"])
def test_record_tp_parity(e3, case):
    """Records against the oracle.  The operand staging decides the rows per
    wave (4, 2 or 1 within 64 KiB of LDS): the l <= 3 input layout runs its
    forward at 4 and its backward at 1, the l <= 2 input layout (106 output
    rows) its dx at 2; R = 57 leaves a ragged last block for each."""
    import torch
    _say("record tp", case)
    rng = np.random.default_rng(61)
    if case == "layout-l2in":
        lay = oirreps.layout("8x0e+8x1o+8x2e", 3, 3)
        i0, i1, i2, v = _layout_records(lay)
        dx_, dy_, dz_ = lay.d_in, lay.d_sh, lay.d_out
        C = 100
    elif case in ("layout-shared", "layout-perchannel", "C7"):
        lay = oirreps.layout("8x0e+8x1o+8x2e+8x3o", 3, 3)
        i0, i1, i2, v = _layout_records(lay)
        dx_, dy_, dz_ = lay.d_in, lay.d_sh, lay.d_out
        C = 7 if case == "C7" else 100
    elif case == "collapsed":
        lay = oirreps.layout("4x0e+4x1o", 2, 1)
        i0, i1, i2, v = _layout_records(lay)
        i0 = np.minimum(i0, 3)   # fold every output row past 3 onto row 3
        dx_, dy_, dz_ = lay.d_in, lay.d_sh, 4
        C = 64
    else:
        dx_, dy_, dz_, nnz = 11, 9, 23, 300
        i0, i1, i2 = rng.integers(0, dz_, nnz), rng.integers(0, dx_, nnz), rng.integers(0, dy_, nnz)
        v = rng.standard_normal(nnz)
        C = 130
    ypc = case.endswith("perchannel") or case == "C7"
    R = 57
    T = e3.RecordTP(dx_, dy_, dz_, i0, i1, i2, v, ypc)
    x = rng.standard_normal((R, dx_, C)).astype(np.float32)
    y = rng.standard_normal((R, dy_, C) if ypc else (R, dy_)).astype(np.float32)
    dz = rng.standard_normal((R, dz_, C)).astype(np.float32)
    vf = v.astype(np.float32).astype(np.float64)
    z = to_np(T.forward(to_dev(x), to_dev(y)))
    gdx, gdy = (to_np(t) for t in T.backward(to_dev(x), to_dev(y), to_dev(dz)))
    rz = ogeneric.tp(i0, i1, i2, vf, x, y, dz_)
    rdx, rdy = ogeneric.tp_bwd(i0, i1, i2, vf, x, y, dz)
    errs = dict(z=rel_l2(z, rz), dx=rel_l2(gdx, rdx), dy=rel_l2(gdy, rdy))
    print("rel-L2", errs, flush=True)
    for k, e in errs.items():
        assert e < TOL, (k, e)


def test_record_tp_200k_rows_matches_specialised(e3):
    """200,000 rows, 128x0e+128x1o+128x2e, l <= 3, with the plan's own records:
    the record kernel against the oracle on sampled rows, and against the
    specialised tensor product on all rows."""
    import torch
    _say("record tp 200k rows")
    cfg = synth.CONFIGS["tp200k"]
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    lay = layout_of(cfg)
    i0, i1, i2, v = _layout_records(lay)
    T = e3.RecordTP(lay.d_in, lay.d_sh, lay.d_out, i0, i1, i2, v, False)
    x, u, w = synth.tp_inputs(cfg)
    y = osh.sh_unit(3, u.astype(np.float64)).astype(np.float32)
    xs, ys = to_dev(x), to_dev(y)
    z = T.forward(xs, ys)
    ones = torch.ones((x.shape[0], plan.P, plan.C), device="cuda")
    zs = e3.tp_fwd(plan, xs, ys, ones)
    torch.cuda.synchronize()
    assert rel_l2(to_np(z), to_np(zs)) < TOL
    rows = np.concatenate([[0, x.shape[0] - 1], np.random.default_rng(62).integers(0, x.shape[0], 30)])
    ri = torch.as_tensor(rows, device="cuda")
    ref = ogeneric.tp(i0, i1, i2, v.astype(np.float32).astype(np.float64), x[rows], y[rows], lay.d_out)
    assert rel_l2(to_np(z[ri]), ref) < TOL


@pytest.mark.parametrize("ypc", [False, True])
def test_record_tp_float64(e3, ypc):
    """The float64 record path against the oracle at float64 accuracy (operand
    rows of up to 64 KiB of doubles per 64 channels; larger ones are refused)."""
    _say("record tp f64", ypc)
    rng = np.random.default_rng(63)
    big = oirreps.layout("4x0e+4x1o+4x2e+4x3o", 3, 3)      # dz rows of 156 doubles: over the limit
    Tb = e3.RecordTP(big.d_in, big.d_sh, big.d_out, *_layout_records(big), ypc)
    with pytest.raises(e3.E3Error) as ei:
        Tb.backward(*(to_dev(np.zeros(sh)) for sh in ((2, big.d_in, 8), (2, big.d_sh, 8) if ypc else (2, big.d_sh),
                                                       (2, big.d_out, 8))))
    assert ei.value.status == 2
    lay = oirreps.layout("4x0e+4x1o+4x2e", 3, 2)
    i0, i1, i2, v = _layout_records(lay)
    R, C = 41, 70
    T = e3.RecordTP(lay.d_in, lay.d_sh, lay.d_out, i0, i1, i2, v, ypc)
    x = rng.standard_normal((R, lay.d_in, C))
    y = rng.standard_normal((R, lay.d_sh, C) if ypc else (R, lay.d_sh))
    dz = rng.standard_normal((R, lay.d_out, C))
    z = to_np(T.forward(to_dev(x), to_dev(y)))
    gdx, gdy = (to_np(t) for t in T.backward(to_dev(x), to_dev(y), to_dev(dz)))
    rz = ogeneric.tp(i0, i1, i2, v, x, y, lay.d_out)
    rdx, rdy = ogeneric.tp_bwd(i0, i1, i2, v, x, y, dz)
    errs = dict(z=rel_l2(z, rz), dx=rel_l2(gdx, rdx), dy=rel_l2(gdy, rdy))
    print("rel-L2", errs, flush=True)
    for k, e in errs.items():
        assert e < 1e-12, (k, e)


def test_conv_step_in_captured_graph(e3):
    """The forward + backward convolution captured in a HIP graph and replayed
    several times, with eager work and synchronisations between replays: every
    replay equals the eager result bit for bit (no allocation, memset or
    synchronisation happens inside the entry points)."""
    import torch
    _say("conv in captured graph")
    rng = np.random.default_rng(71)
    irreps = "128x0e+128x1o+128x2e+128x3o"
    lay = oirreps.layout(irreps, 3, 3)
    n, e = 300, 6000
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    plan = e3.Plan(irreps, 3, 3)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n)
    xs = to_dev(rng.standard_normal((n, lay.d_in, C)).astype(np.float32))
    vs = to_dev(vec)
    ss = to_dev(rng.standard_normal((e, lay.n_paths, C)).astype(np.float32))
    dms = to_dev(rng.standard_normal((n, lay.d_out, C)).astype(np.float32))
    ws = e3.workspace(e3.conv_workspace_size(plan, G)[1])
    m = torch.empty((n, lay.d_out, C), device="cuda")
    dx = torch.empty_like(xs)
    dvec = torch.empty_like(vs)
    ds = torch.empty_like(ss)

    def step():
        e3.conv_fwd(plan, G, xs, vs, ss, out=m)
        e3.conv_bwd(plan, G, xs, vs, ss, dms, dx=dx, dvec=dvec, ds=ds, ws=ws)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (m, dx, dvec, ds)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for it in range(4):
        for t in (m, dx, dvec, ds):
            t.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip((m, dx, dvec, ds), ref):
            assert torch.equal(a, b), it
        # eager work between replays, on the same buffers' inputs
        _ = e3.conv_fwd(plan, G, xs, vs, ss)
        torch.cuda.synchronize()



def test_extensions_in_captured_graph(e3):
    """The double backward, the fused-radial forward and backward and the
    tensor product forward and backward captured in one HIP graph and replayed
    several times, with eager work between replays: every replay equals the
    eager result bit for bit."""
    import torch
    _say("extensions in captured graph")
    rng = np.random.default_rng(72)
    irreps = "128x0e+128x1o+128x2e+128x3o"
    lay = oirreps.layout(irreps, 3, 3)
    n, e, K, R = 200, 3000, 8, 500
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    plan = e3.Plan(irreps, 3, 3)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=5)
    f = lambda *shape: to_dev(rng.standard_normal(shape).astype(np.float32))
    x, vs, s, dm = f(n, lay.d_in, C), to_dev(vec), f(e, lay.n_paths, C), f(n, lay.d_out, C)
    y, ddx, ddy, dds = f(e, lay.d_sh), f(n, lay.d_in, C), f(e, lay.d_sh), f(e, lay.n_paths, C)
    h, W = f(e, K), f(K, lay.n_paths, C)
    tx, ty, tw, tdz = f(R, lay.d_in, C), f(R, lay.d_sh), f(R, lay.n_paths, C), f(R, lay.d_out, C)
    ws2 = e3.workspace(e3.conv_workspace_size(plan, G)[1])
    wsr = e3.workspace(e3.conv_radial_workspace_size(plan, G, K))
    wst = e3.workspace(e3.tp_workspace_size(plan, R))
    m = torch.empty((n, lay.d_out, C), device="cuda")
    rdx, rdvec, rdh, rdW = (torch.empty_like(t) for t in (x, vs, h, W))
    tz = torch.empty_like(tdz)
    tdx, tdy, tdw = torch.empty_like(tx), torch.empty_like(ty), torch.empty_like(tw)
    outs = {}

    def step():
        outs["bwd2"] = e3.conv_bwd2(plan, G, x, y, s, dm, ddx, ddy, dds, ws=ws2)
        e3.conv_fwd_radial(plan, G, x, vs, h, W, out=m)
        e3.conv_bwd_radial(plan, G, x, vs, h, W, dm, dx=rdx, dvec=rdvec, dh=rdh, dW=rdW, ws=wsr)
        e3.tp_fwd(plan, tx, ty, tw, out=tz)
        e3.tp_bwd(plan, tx, ty, tw, tdz, tdx, tdy, tdw, wst)

    def results():
        return list(outs["bwd2"]) + [m, rdx, rdvec, rdh, rdW, tz, tdx, tdy, tdw]

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in results()]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for it in range(3):
        for t in results():
            t.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(results(), ref):
            assert torch.equal(a, b), it
        _ = e3.conv_fwd(plan, G, x, vs, s)   # eager work between replays
        torch.cuda.synchronize()


def test_conv_on_side_stream(e3):
    """Forward + backward launched on a stream other than torch's current one:
    outputs and workspace are allocated for that stream, and the results equal
    those of the current stream bit for bit, also with a large allocation made
    on the current stream while the side stream's kernels may still run."""
    import torch
    _say("conv on a side stream")
    rng = np.random.default_rng(72)
    irreps = "128x0e+128x1o+128x2e+128x3o"
    lay = oirreps.layout(irreps, 3, 3)
    n, e = 400, 9000
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    plan = e3.Plan(irreps, 3, 3)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n)
    xs = to_dev(rng.standard_normal((n, lay.d_in, C)).astype(np.float32))
    vs = to_dev(vec)
    ss = to_dev(rng.standard_normal((e, lay.n_paths, C)).astype(np.float32))
    dms = to_dev(rng.standard_normal((n, lay.d_out, C)).astype(np.float32))
    ref = [e3.conv_fwd(plan, G, xs, vs, ss), *e3.conv_bwd(plan, G, xs, vs, ss, dms)]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        m = e3.conv_fwd(plan, G, xs, vs, ss, stream=side)
        dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, ss, dms, stream=side)
        junk = torch.full((64 << 20,), float("nan"), device="cuda")   # current stream
        torch.cuda.current_stream().wait_stream(side)
        for a, b in zip((m, dx, dvec, ds), ref):
            assert torch.equal(a, b)
        del junk
    torch.cuda.synchronize()



def test_linear_and_record_descriptors(e3):
    """Descriptor sizes against the oracle's plan, and the argument checks of
    the compute calls; a valid descriptor uploads its tables when created."""
    import ctypes as ct
    _say("linear and record descriptors")
    for ins, outs in [("16x0e+16x1o+16x1o+16x2e", "32x0e+32x1o+32x1e+32x2e"),
                      ("128x0e+128x1o+128x2e+128x3o", "128x0e+128x1o+128x2e+128x3o")]:
        L = e3.Linear(ins, outs)
        jobs, d_in, d_out, c_in, c_out, nw = olinear.plan(ins, outs)
        assert (L.n_weights, L.D_in, L.D_out, L.C_in, L.C_out) == (nw, d_in, d_out, c_in, c_out)
        L.close()
    L = e3.Linear("16x0e", "16x0e")
    Ll = e3.lib()
    assert Ll.e3_linear_fwd(L.handle, None, None, None, -1, None) == 1
    assert Ll.e3_linear_fwd(L.handle, None, None, None, 0, None) == 0
    assert Ll.e3_linear_fwd(L.handle, None, None, None, 5, None) == 1
    n = ct.c_size_t()
    assert Ll.e3_linear_workspace_size(L.handle, ct.byref(n)) == 0 and n.value > 0
    assert Ll.e3_linear_bwd(L.handle, None, None, None, None, None, None, 0, 5, None) == 1
    L.close()
    h = ct.c_void_p()
    i = (ct.c_int32 * 2)(0, 1)
    v = (ct.c_double * 2)(1.0, 2.0)
    assert Ll.e3_tpg_create(4, 4, 4, 2, i, i, i, v, 1, ct.byref(h)) == 0
    assert Ll.e3_tpg_destroy(h) == 0
    assert Ll.e3_tpg_create(4, 4, 4, 0, None, None, None, None, 0, ct.byref(h)) == 0
    assert Ll.e3_tpg_workspace_size(h, 10, 128, ct.byref(n)) == 0 and n.value >= 10 * 2 * 4 * 4
    assert Ll.e3_tpg_fwd(h, None, None, None, 0, 8, None) == 0
    assert Ll.e3_tpg_fwd(h, None, None, None, 3, 8, None) == 1
    assert Ll.e3_tpg_destroy(h) == 0


def test_first_linear_and_record_calls_in_captured_graph(e3):
    """A linear mixing and a record tensor product whose very first forward
    calls are made under HIP graph capture (their tables were uploaded when the
    descriptors were created, so the calls only launch kernels): every replay
    equals the eager result bit for bit and the oracle to the parity bar."""
    import torch
    _say("first linear / record calls in a captured graph")
    rng = np.random.default_rng(73)
    ins, outs, n = "32x0e+32x1o+32x1o", "32x0e+32x1o", 300
    L = e3.Linear(ins, outs)
    x = rng.standard_normal((n, L.D_in, L.C_in)).astype(np.float32)
    W = (rng.standard_normal(L.n_weights) / 8).astype(np.float32)
    xs, Ws = to_dev(x), to_dev(W)
    lay = oirreps.layout("64x0e+64x1o", 2, 2)
    recs = ocg.coo_records(lay)
    i0, i1, i2, rv = (np.array([r[k] for r in recs]) for k in range(4))
    R = e3.RecordTP(lay.d_in, lay.d_sh, lay.d_out, i0, i1, i2, rv, False)
    rows = 500
    xr = rng.standard_normal((rows, lay.d_in, lay.channels)).astype(np.float32)
    yr = rng.standard_normal((rows, lay.d_sh)).astype(np.float32)
    xrs, yrs = to_dev(xr), to_dev(yr)
    out = torch.empty((n, L.D_out, L.C_out), device="cuda")
    zr = torch.empty((rows, lay.d_out, lay.channels), device="cuda")
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        L.forward(xs, Ws, out=out)
        R.forward(xrs, yrs, out=zr)
    torch.cuda.synchronize()
    ref_out = L.forward(xs, Ws)
    ref_z = R.forward(xrs, yrs)
    torch.cuda.synchronize()
    assert rel_l2(to_np(ref_out), olinear.forward(ins, outs, x, W).numpy()) < TOL
    assert rel_l2(to_np(ref_z), ogeneric.tp(i0, i1, i2, rv, xr, yr, lay.d_out)) < TOL
    for it in range(3):
        out.fill_(float("nan"))
        zr.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref_out) and torch.equal(zr, ref_z), it
        _ = L.forward(xs, Ws)
        torch.cuda.synchronize()
    L.close()
    R.close()



# ---------------------------------------------------------------- float64 builds
# Bar for the float64 kernels, derived from the arithmetic: one float64 rounding
# per term (about 1.1e-16) grown by the square root of the terms summed (a few
# hundred per output here, so about 3e-15) and by the cancellation a random-sign
# sum can add; 1e-12 leaves ample margin.
TOL64 = 1e-12


@pytest.mark.parametrize("case", ["cube64", "random_l3_pad", "natural_l3", "reordered_l3"])
def test_conv_float64(e3, case):
    """The float64 build of the convolution (forward, dx, ds, dvec) against the
    fp64 oracle on the same float64 inputs, and the float32 build's error
    measured against it, as the paper compares its kernels' precisions."""
    import torch
    _say("conv float64", case)
    rng = np.random.default_rng(21)
    if case == "cube64":
        cfg = synth.CONFIGS["cube64"]
        g = synth.graph(cfg)
        snd, rcv, n, vec = g.sender, g.receiver, g.n_nodes, g.vec.astype(np.float64)
        irreps, lsh, lout, parity, pad = cfg.irreps, cfg.lmax_sh, cfg.lmax_out, "all", -1
    else:
        irreps = {"random_l3_pad": "64x0e+64x1o+64x2e+64x3o", "natural_l3": "32x0e+32x1o+32x2e+32x3o",
                  "reordered_l3": "16x1o+16x0e+16x3o+16x2e"}[case]
        parity = "natural" if case == "natural_l3" else "all"
        lsh = lout = 3
        n, e = 70, 1300
        pad = 5 if case == "random_l3_pad" else -1
        snd, rcv, vec32 = _random_graph(rng, n, e)
        vec = rng.standard_normal((e, 3)) * 2.0
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = e3.Plan(irreps, lsh, lout, natural=parity == "natural")
    E, C = snd.shape[0], lay.channels
    x = rng.standard_normal((n, lay.d_in, C))
    s = rng.standard_normal((E, lay.n_paths, C))
    dm = rng.standard_normal((n, lay.d_out, C))
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    d64 = [torch.from_numpy(a).to("cuda") for a in (x, vec, s, dm)]
    m = e3.conv_fwd_f64(plan, G, *d64[:3])
    dx, dvec, ds = e3.conv_bwd_f64(plan, G, *d64)
    torch.cuda.synchronize()
    ref_m = oconv.conv_fwd(lay, x, vec, s, snd, rcv, n, pad_node=pad).numpy()
    ref = oconv.conv_bwd(lay, x, vec, s, dm, snd, rcv, n, pad_node=pad)
    refs = dict(m=ref_m, dx=ref["dx"].numpy(), ds=ref["ds"].numpy(), dvec=ref["dvec"].numpy())
    got = dict(m=m, dx=dx, ds=ds, dvec=dvec)
    errs = {k: rel_l2(to_np(got[k]), refs[k]) for k in refs}
    print("float64 rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL64, (k, v)
    # the float32 build on the same inputs rounded to float32, against float64
    d32 = [t.float() for t in d64]
    m32 = e3.conv_fwd(plan, G, *d32[:3])
    dx32, dvec32, ds32 = e3.conv_bwd(plan, G, *d32)
    e32 = dict(m=rel_l2(to_np(m32), refs["m"]), dx=rel_l2(to_np(dx32), refs["dx"]),
               ds=rel_l2(to_np(ds32), refs["ds"]), dvec=rel_l2(to_np(dvec32), refs["dvec"]))
    print("float32 rel-L2 against float64", e32, flush=True)
    for k, v in e32.items():
        assert v < TOL, (k, v)
    again = e3.conv_bwd_f64(plan, G, *d64)
    for a, b in zip((dx, dvec, ds), again):
        assert torch.equal(a, b)


@pytest.mark.parametrize("irreps,lsh,lout,parity,rows", [
    ("128x0e+128x1o+128x2e", 3, 3, "all", 61),     # the 200k-row layout
    ("8x0e+8x1o", 2, 2, "all", 5),
    ("96x0e+96x1o+96x2e+96x3o", 3, 3, "natural", 17),
])
def test_tp_float64(e3, irreps, lsh, lout, parity, rows):
    """The float64 build of the weighted tensor product and its backward."""
    import torch
    _say("tp float64", irreps, parity, rows)
    rng = np.random.default_rng(22)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = e3.Plan(irreps, lsh, lout, natural=parity == "natural")
    C = lay.channels
    x = rng.standard_normal((rows, lay.d_in, C))
    g = rng.standard_normal((rows, 3))
    y = osh.sh_unit(lsh, g / np.linalg.norm(g, axis=1, keepdims=True))
    w = rng.standard_normal((rows, lay.n_paths, C))
    dz = rng.standard_normal((rows, lay.d_out, C))
    dev = [torch.from_numpy(np.ascontiguousarray(a)).to("cuda") for a in (x, y, w, dz)]
    z = e3.tp_fwd_f64(plan, *dev[:3])
    dx, dy, dw = e3.tp_bwd_f64(plan, *dev)
    torch.cuda.synchronize()
    errs = dict(z=rel_l2(to_np(z), otp.tp(lay, x, y, w).numpy()))
    for k, a, r in zip(("dx", "dy", "dw"), (dx, dy, dw), otp.tp_bwd(lay, x, y, w, dz)):
        errs[k] = rel_l2(to_np(a), r.numpy())
    print("float64 rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL64, (k, v)


def test_probe_stream_bytes_and_writes(e3):
    """The streaming probe moves exactly the bytes it reports, writes every
    unit of the destination it covers (the step index mod 1024, one value per
    unit) and leaves the rest alone; its launch is timed."""
    import torch
    _say("probe stream")
    dev = torch.device("cuda")
    src = torch.ones(1 << 18, dtype=torch.float32, device=dev)          # 1 MiB
    dst = torch.full((1 << 18,), -1.0, dtype=torch.float32, device=dev)
    e3.timing_reset()
    e3.timing_enable(True)
    br, bw = e3.probe_stream(src, dst, 2, 6, 8, 3)
    torch.cuda.synchronize()
    e3.timing_enable(False)
    unit = 64 * 8
    steps = min((1 << 20) // (2 * unit), (1 << 20) // (6 * unit))
    assert (br, bw) == (steps * 2 * unit, steps * 6 * unit)
    got = to_np(dst).reshape(-1)
    per_step = 6 * unit // 4
    for st in (0, 1, steps // 2, steps - 1):
        assert np.all(got[st * per_step:(st + 1) * per_step] == float(st & 1023)), st
    assert np.all(got[steps * per_step:] == -1.0)
    assert "probe_stream" in e3.timing_read()
    br, bw = e3.probe_stream(src, None, 16, 0, 16, 1)
    torch.cuda.synchronize()
    assert bw == 0 and br == (1 << 20) // (16 * 64 * 16) * 16 * 64 * 16


# ---------------------------------------------------------------- capacity (last: largest)
def test_conv_stress_water70k_sampled(e3):
    """70,000 H2O (210,000 atoms, ~11M edges), 64 channels: forward + backward at
    full size on one GPU, checked on sampled rows.  Last in the file: it takes
    most of the GPU's memory (about 250 GB) and the longest time."""
    import torch
    _say("conv stress water70k")
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    cfg = synth.CONFIGS["water70k"]
    g = synth.graph(cfg)
    N, E = g.n_nodes, g.sender.shape[0]
    print(f"N={N} E={E}", flush=True)
    plan = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    dev = torch.device("cuda")
    x = synth.node_features(cfg, N)
    s = synth.normal_device(cfg.cid, 2, (E, plan.P, plan.C), dev)
    dm = synth.normal_device(cfg.cid, 3, (N, plan.D_out, plan.C), dev)
    G = e3.Graph(to_dev(g.sender), to_dev(g.receiver), N)
    xs, vs = to_dev(x), to_dev(g.vec)
    m = e3.conv_fwd(plan, G, xs, vs, s)
    torch.cuda.synchronize()
    lay = layout_of(cfg)
    rng = np.random.default_rng(9)
    rs = np.concatenate([[0, N - 1], rng.choice(N, 14, replace=False)])
    es = np.concatenate([[0, E - 1], rng.choice(E, 30, replace=False)])
    sfn = lambda rows: s[torch.as_tensor(rows, device=dev)].cpu().numpy()
    ref_m = oracle_fwd_rows(lay, x, g.vec, sfn, g.sender, g.receiver, N, rs)
    err_m = rel_l2(to_np(m[torch.as_tensor(rs, device=dev)]), ref_m)
    del m
    torch.cuda.empty_cache()
    dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, s, dm)
    torch.cuda.synchronize()
    ref_dx, ref_ds, ref_dv = oracle_bwd_rows(lay, x, g.vec, sfn, dm, g.sender, g.receiver, N, rs, es)
    ri, ei = torch.as_tensor(rs, device=dev), torch.as_tensor(es, device=dev)
    errs = dict(m=err_m, dx=rel_l2(to_np(dx[ri]), ref_dx), ds=rel_l2(to_np(ds[ei]), ref_ds),
                dvec=rel_l2(to_np(dvec[ei]), ref_dv))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    del dx, dvec, ds, s, dm, G
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
