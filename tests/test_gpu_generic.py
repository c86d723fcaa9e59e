"""GPU parity of the two paths for layouts without compiled kernels -- the
composed path (generated single-block kinds run block by block) and the
record path (the plan's coupling records walked at run time) -- on such
layouts and on compiled ones forced onto them, against the fp64 oracle.

Bar: relative L2 <= 1e-5 per output tensor; padding rows exactly zero;
bitwise-identical repeats.
"""
import numpy as np
import pytest

import synth
from oracle import conv as oconv
from oracle import irreps as oirreps
from oracle import radial as oradial
from oracle import sh as osh
from oracle import tp as otp

from gpu_util import TOL, layout_of, oracle_bwd_rows, oracle_fwd_rows, rel_l2, to_dev, to_np, upload_weights

pytestmark = pytest.mark.gpu

TOL64 = 1e-12   # float64 builds against the float64 oracle (the bar of the compiled float64 tests)


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


def _random_graph(rng, n, e):
    snd = rng.integers(0, n, e).astype(np.int32)
    rcv = rng.integers(0, n, e).astype(np.int32)
    rcv = np.where(rcv == snd, (rcv + 1) % n, rcv).astype(np.int32)
    vec = (rng.standard_normal((e, 3)) * 2.0).astype(np.float32)
    return snd, rcv, vec


PATHS = ["composed", "records"]


def _plan(e3, irreps, lsh, lout, parity, path):
    plan = e3.Plan(irreps, lsh, lout, natural=parity == "natural", records=path == "records",
                   composed=path == "composed")
    assert plan.kernels == path, (irreps, plan.kernels)
    return plan


# (irreps, lmax_sh, lmax_out, parity, n, e, pad)
CASES = [
    ("16x0e+16x0o+16x1o+16x1e", 2, 2, "all", 50, 700, -1),   # two blocks of each degree
    ("32x2e+32x0e+32x1o", 3, 3, "all", 60, 900, 5),          # blocks out of degree order
    ("8x3o+8x1e", 1, 3, "natural", 40, 500, -1),             # natural parities, l_sh 1
    ("68x1o+68x2o", 3, 2, "all", 45, 600, 3),                # a ragged second channel slab
    ("4x0e", 0, 0, "all", 30, 200, -1),                      # the smallest layout
    ("8x0o+8x1o", 1, 1, "natural", 40, 500, 2),              # a block with no path
    ("1024x1o+1024x1e", 1, 1, "all", 10, 60, -1),            # 16 channel slabs
    ("128x0e+128x1o+128x2e+128x3o", 2, 3, "all", 60, 1200, -1),
    ("64x0e+64x1o+64x1e+64x2e+64x3o", 3, 3, "natural", 40, 600, 4),
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, "all", 80, 1500, 7),   # the benchmark layout (compiled too)
    ("12x0e+12x1o+12x2e+12x3o+12x0o+12x1e+12x2o+12x3e", 3, 3, "all", 30, 400, -1),   # eight blocks
]


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("irreps,lsh,lout,parity,n,e,pad", CASES)
def test_generic_conv_full(e3, irreps, lsh, lout, parity, n, e, pad, path):
    import torch
    _say("generic conv", path, irreps, lsh, lout, parity, n, e, pad)
    rng = np.random.default_rng(41)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = _plan(e3, irreps, lsh, lout, parity, path)
    assert (plan.P, plan.D_out) == (lay.n_paths, lay.d_out)
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
    s = rng.standard_normal((e, lay.n_paths, C)).astype(np.float32)
    dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    xs, vs, ss, dms = to_dev(x), to_dev(vec), to_dev(s), to_dev(dm)
    outs = []
    for _ in range(2):
        m = e3.conv_fwd(plan, G, xs, vs, ss)
        dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, ss, dms)
        outs.append((m, dx, dvec, ds))
    torch.cuda.synchronize()
    for a, b in zip(*outs):
        assert torch.equal(a, b)
    m, dx, dvec, ds = outs[0]
    ref_m = oconv.conv_fwd(lay, x, vec, s, snd, rcv, n, pad_node=pad).numpy()
    ref = oconv.conv_bwd(lay, x, vec, s, dm, snd, rcv, n, pad_node=pad)
    errs = dict(m=rel_l2(to_np(m), ref_m), dx=rel_l2(to_np(dx), ref["dx"].numpy()),
                ds=rel_l2(to_np(ds), ref["ds"].numpy()), dvec=rel_l2(to_np(dvec), ref["dvec"].numpy()))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    if pad >= 0:
        dead = (snd == pad) | (rcv == pad)
        assert np.all(to_np(ds)[dead] == 0) and np.all(to_np(dvec)[dead] == 0)
        assert np.all(to_np(m)[pad] == 0) and np.all(to_np(dx)[pad] == 0)
    cp = e3.Plan(irreps, lsh, lout, natural=parity == "natural")
    if cp.kernels == "compiled":  # the compiled kernels of the same layout agree to rounding
        mc = e3.conv_fwd(cp, G, xs, vs, ss)
        dxc, dvc, dsc = e3.conv_bwd(cp, G, xs, vs, ss, dms)
        for a, b in ((m, mc), (dx, dxc), (dvec, dvc), (ds, dsc)):
            assert rel_l2(to_np(a), to_np(b)) < 1e-6


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("irreps,lsh,lout,parity,rows", [
    ("16x0e+16x0o+16x1o+16x1e", 2, 2, "all", 37),
    ("68x1o+68x2o", 3, 2, "all", 300),
    ("8x0o+8x1o", 1, 1, "natural", 50),
    ("32x0e+32x1o+32x2e", 2, 2, "all", 257),
])
def test_generic_tp_fwd_bwd(e3, irreps, lsh, lout, parity, rows, path):
    """The weighted tensor product on the composed path (single-block tensor
    product kernels) and on the record path (the convolution code on the
    identity graph), forward and backward, against the oracle."""
    _say("generic tp", path, irreps, lsh, lout, parity, rows)
    rng = np.random.default_rng(42)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = _plan(e3, irreps, lsh, lout, parity, path)
    C = lay.channels
    g = rng.standard_normal((rows, 3))
    y = osh.sh_unit(lsh, g / np.linalg.norm(g, axis=1, keepdims=True)).astype(np.float32)
    x = rng.standard_normal((rows, lay.d_in, C)).astype(np.float32)
    w = rng.standard_normal((rows, lay.n_paths, C)).astype(np.float32)
    dz = rng.standard_normal((rows, lay.d_out, C)).astype(np.float32)
    z = to_np(e3.tp_fwd(plan, to_dev(x), to_dev(y), to_dev(w)))
    assert rel_l2(z, otp.tp(lay, x, y, w).numpy()) < TOL
    got = [to_np(t) for t in e3.tp_bwd(plan, to_dev(x), to_dev(y), to_dev(w), to_dev(dz))]
    for name, a, r in zip(("dx", "dy", "dw"), got, otp.tp_bwd(lay, x, y, w, dz)):
        err = rel_l2(a, r.numpy())
        print(name, err, flush=True)
        assert err < TOL, name


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("irreps,lsh,lout,parity,n,e,pad", [
    ("16x0e+16x0o+16x1o+16x1e", 2, 2, "all", 40, 600, -1),
    ("68x1o+68x2o", 3, 2, "all", 30, 400, 4),
    ("8x0o+8x1o", 1, 1, "natural", 30, 400, -1),
])
def test_generic_conv_y_accumulate_optional(e3, irreps, lsh, lout, parity, n, e, pad, path):
    """Caller harmonics y, accumulation and omitted cotangents."""
    import torch
    _say("generic conv y-input", path, irreps, n, e, pad)
    rng = np.random.default_rng(43)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = _plan(e3, irreps, lsh, lout, parity, path)
    snd, rcv, _ = _random_graph(rng, n, e)
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
    y = rng.standard_normal((e, lay.d_sh)).astype(np.float32)
    s = rng.standard_normal((e, lay.n_paths, C)).astype(np.float32)
    dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
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
    m2 = m.clone()
    e3.conv_fwd_y(plan, G, xs, ys, ss, out=m2, accumulate=True)
    d2 = [t.clone() for t in (dx, dy, ds)]
    e3.conv_bwd_y(plan, G, xs, ys, ss, dms, dx=d2[0], dy=d2[1], ds=d2[2], accumulate=True)
    assert torch.equal(m2, 2 * m)
    for a, b in zip(d2, (dx, dy, ds)):
        assert torch.equal(a, 2 * b)
    for want in (("dx",), ("dy",), ("ds",), ("dy", "ds")):
        got = e3.conv_bwd_y(plan, G, xs, ys, ss, dms, want=want)
        for name, full, part in zip(("dx", "dy", "ds"), (dx, dy, ds), got):
            if name in want:
                assert torch.equal(full, part), (want, name)
            else:
                assert part is None


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("irreps,lsh,lout,parity,n,e,pad", [
    ("16x0e+16x0o+16x1o+16x1e", 2, 2, "all", 30, 400, -1),
    ("32x2e+32x0e+32x1o", 3, 3, "all", 25, 300, 3),
    ("132x1o+132x0e+132x2e", 2, 2, "all", 20, 250, -1),  # three channel slabs, the last of four channels
])
def test_generic_conv_bwd2(e3, irreps, lsh, lout, parity, n, e, pad, path):
    """Double backward (three forward and three backward passes) against the
    oracle."""
    import torch
    _say("generic conv bwd2", path, irreps, n, e, pad)
    rng = np.random.default_rng(44)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = _plan(e3, irreps, lsh, lout, parity, path)
    snd, rcv, _ = _random_graph(rng, n, e)
    C = lay.channels
    arrs = dict(x=(n, lay.d_in, C), y=(e, lay.d_sh), s=(e, lay.n_paths, C), dm=(n, lay.d_out, C),
                ddx=(n, lay.d_in, C), ddy=(e, lay.d_sh), dds=(e, lay.n_paths, C))
    a = {k: rng.standard_normal(v).astype(np.float32) for k, v in arrs.items()}
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


@pytest.mark.parametrize("path", PATHS)
def test_generic_conv_degenerate_graphs(e3, path):
    """No edges; a single edge; nodes without in-edges."""
    irreps, lsh, lout = "16x0e+16x0o+16x1o+16x1e", 2, 2
    lay = oirreps.layout(irreps, lsh, lout)
    plan = _plan(e3, irreps, lsh, lout, "all", path)
    C = lay.channels
    rng = np.random.default_rng(45)
    for snd, rcv, n in [(np.zeros(0, np.int32), np.zeros(0, np.int32), 4),
                        (np.array([2], np.int32), np.array([0], np.int32), 3)]:
        _say("generic conv degenerate", path, len(snd))
        e = len(snd)
        vec = rng.standard_normal((e, 3)).astype(np.float32)
        x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
        s = rng.standard_normal((e, lay.n_paths, C)).astype(np.float32)
        dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
        G = e3.Graph(to_dev(snd), to_dev(rcv), n)
        xs, vs, ss, dms = to_dev(x), to_dev(vec), to_dev(s), to_dev(dm)
        m = e3.conv_fwd(plan, G, xs, vs, ss)
        dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, ss, dms)
        if e == 0:
            assert np.all(to_np(m) == 0) and np.all(to_np(dx) == 0)
        else:
            ref_m = oconv.conv_fwd(lay, x, vec, s, snd, rcv, n).numpy()
            ref = oconv.conv_bwd(lay, x, vec, s, dm, snd, rcv, n)
            assert rel_l2(to_np(m), ref_m) < TOL
            assert rel_l2(to_np(dx), ref["dx"].numpy()) < TOL
            assert rel_l2(to_np(ds), ref["ds"].numpy()) < TOL
            assert rel_l2(to_np(dvec), ref["dvec"].numpy()) < TOL
            assert np.all(to_np(m)[1:] == 0)


@pytest.mark.parametrize("path", PATHS)
def test_generic_conv_water8k_sampled(e3, path):
    """The benchmark workload (24,000-atom water box, 128x0e+128x1o+128x2e+128x3o,
    l <= 3) forced onto each path at full size: sampled receivers, senders and
    edges against the oracle, and the whole outputs against the compiled
    kernels."""
    _say("generic conv water8k", path)
    cfg = synth.CONFIGS["water8k"]
    g = synth.graph(cfg)
    x = synth.node_features(cfg, g.n_nodes)
    dm = synth.out_cotangent(cfg, g.n_nodes)
    plan = _plan(e3, cfg.irreps, cfg.lmax_sh, cfg.lmax_out, "all", path)
    s = upload_weights(cfg, g.vec)
    G = e3.Graph(to_dev(g.sender), to_dev(g.receiver), g.n_nodes)
    xs, vs, dms = to_dev(x), to_dev(g.vec), to_dev(dm)
    m = e3.conv_fwd(plan, G, xs, vs, s)
    dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, s, dms)
    lay = layout_of(cfg)
    rng = np.random.default_rng(46)
    rs = rng.choice(g.n_nodes, 24, replace=False)
    es = rng.choice(g.sender.shape[0], 64, replace=False)
    W = synth.bessel_matrix(cfg)
    sfn = lambda rows: synth.edge_weights_rows(cfg, g.vec, rows, W=W)
    ref_m = oracle_fwd_rows(lay, x, g.vec, sfn, g.sender, g.receiver, g.n_nodes, rs)
    ref_dx, ref_ds, ref_dv = oracle_bwd_rows(lay, x, g.vec, sfn, dm, g.sender, g.receiver, g.n_nodes, rs, es)
    import torch
    ri, ei = torch.as_tensor(rs, device="cuda"), torch.as_tensor(es, device="cuda")
    errs = dict(m=rel_l2(to_np(m[ri]), ref_m), dx=rel_l2(to_np(dx[ri]), ref_dx),
                ds=rel_l2(to_np(ds[ei]), ref_ds), dvec=rel_l2(to_np(dvec[ei]), ref_dv))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    cp = e3.Plan(cfg.irreps, cfg.lmax_sh, cfg.lmax_out)
    mc = e3.conv_fwd(cp, G, xs, vs, s)
    dxc, dvc, dsc = e3.conv_bwd(cp, G, xs, vs, s, dms)
    for a, b in ((m, mc), (dx, dxc), (dvec, dvc), (ds, dsc)):
        num = float(torch.linalg.vector_norm((a - b).double()))
        den = float(torch.linalg.vector_norm(b.double()))
        assert num <= 1e-6 * den, (num, den)


def test_generic_paths_in_captured_graph(e3):
    """Both paths only launch kernels: the composed path's convolution forward,
    backward and double backward and tensor product forward and backward, and
    the record path's convolution forward and backward, captured in one HIP
    graph and replayed several times with eager work between replays, equal
    the eager results bit for bit."""
    import torch
    _say("generic paths in captured graph")
    rng = np.random.default_rng(47)
    irreps, lsh, lout = "32x2e+32x0e+32x1o", 3, 3
    lay = oirreps.layout(irreps, lsh, lout)
    cp = _plan(e3, irreps, lsh, lout, "all", "composed")
    rp = _plan(e3, irreps, lsh, lout, "all", "records")
    n, e, R = 150, 2000, 300
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=4)
    f = lambda *shape: to_dev(rng.standard_normal(shape).astype(np.float32))
    x, vs, s, dm = f(n, lay.d_in, C), to_dev(vec), f(e, lay.n_paths, C), f(n, lay.d_out, C)
    y, ddx, ddy, dds = f(e, lay.d_sh), f(n, lay.d_in, C), f(e, lay.d_sh), f(e, lay.n_paths, C)
    tx, ty, tw, tdz = f(R, lay.d_in, C), f(R, lay.d_sh), f(R, lay.n_paths, C), f(R, lay.d_out, C)
    wsc = e3.workspace(e3.conv_workspace_size(cp, G)[1])
    wsr = e3.workspace(e3.conv_workspace_size(rp, G)[1])
    wst = e3.workspace(e3.tp_workspace_size(cp, R))
    m, mr = (torch.empty((n, lay.d_out, C), device="cuda") for _ in range(2))
    dx, dxr = torch.empty_like(x), torch.empty_like(x)
    dvec, dvecr = torch.empty_like(vs), torch.empty_like(vs)
    ds, dsr = torch.empty_like(s), torch.empty_like(s)
    tz = torch.empty_like(tdz)
    tdx, tdy, tdw = torch.empty_like(tx), torch.empty_like(ty), torch.empty_like(tw)
    outs = {}

    def step():
        e3.conv_fwd(cp, G, x, vs, s, out=m)
        e3.conv_bwd(cp, G, x, vs, s, dm, dx=dx, dvec=dvec, ds=ds, ws=wsc)
        outs["bwd2"] = e3.conv_bwd2(cp, G, x, y, s, dm, ddx, ddy, dds, ws=wsc)
        e3.tp_fwd(cp, tx, ty, tw, out=tz)
        e3.tp_bwd(cp, tx, ty, tw, tdz, tdx, tdy, tdw, wst)
        e3.conv_fwd(rp, G, x, vs, s, out=mr)
        e3.conv_bwd(rp, G, x, vs, s, dm, dx=dxr, dvec=dvecr, ds=dsr, ws=wsr)

    def results():
        return [m, dx, dvec, ds] + list(outs["bwd2"]) + [tz, tdx, tdy, tdw, mr, dxr, dvecr, dsr]

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
        _ = e3.conv_fwd(cp, G, x, vs, s)   # eager work between replays
        torch.cuda.synchronize()


@pytest.mark.parametrize("irreps,lsh,lout,parity,n,e,pad,rows", [
    ("16x0e+16x0o+16x1o+16x1e", 2, 2, "all", 50, 700, 3, 37),
    ("8x0o+8x1o", 1, 1, "natural", 40, 500, -1, 20),                # a block with no path
    ("68x1o+68x2o", 3, 2, "all", 30, 400, -1, 11),                  # a ragged second slab
    ("64x0e+64x1o+64x2e+64x3o", 3, 3, "all", 40, 600, 4, 9),        # a compiled layout, forced
])
def test_composed_float64(e3, irreps, lsh, lout, parity, n, e, pad, rows):
    """The float64 builds of the convolution and the tensor product on the
    composed path against the oracle on the same float64 inputs (bar 1e-12),
    with bitwise repeats."""
    import torch
    _say("composed float64", irreps, lsh, lout, parity, n, e, pad, rows)
    rng = np.random.default_rng(48)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = _plan(e3, irreps, lsh, lout, parity, "composed")
    snd, rcv, _ = _random_graph(rng, n, e)
    vec = rng.standard_normal((e, 3)) * 2.0
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C))
    s = rng.standard_normal((e, lay.n_paths, C))
    dm = rng.standard_normal((n, lay.d_out, C))
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    d64 = [torch.from_numpy(a).to("cuda") for a in (x, vec, s, dm)]
    m = e3.conv_fwd_f64(plan, G, *d64[:3])
    dx, dvec, ds = e3.conv_bwd_f64(plan, G, *d64)
    torch.cuda.synchronize()
    ref_m = oconv.conv_fwd(lay, x, vec, s, snd, rcv, n, pad_node=pad).numpy()
    ref = oconv.conv_bwd(lay, x, vec, s, dm, snd, rcv, n, pad_node=pad)
    errs = dict(m=rel_l2(to_np(m), ref_m), dx=rel_l2(to_np(dx), ref["dx"].numpy()),
                ds=rel_l2(to_np(ds), ref["ds"].numpy()), dvec=rel_l2(to_np(dvec), ref["dvec"].numpy()))
    print("float64 conv rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL64, (k, v)
    if pad >= 0:
        dead = (snd == pad) | (rcv == pad)
        assert np.all(to_np(ds)[dead] == 0) and np.all(to_np(dvec)[dead] == 0)
    again = e3.conv_bwd_f64(plan, G, *d64)
    for a, b in zip((dx, dvec, ds), again):
        assert torch.equal(a, b)
    g = rng.standard_normal((rows, 3))
    y = osh.sh_unit(lsh, g / np.linalg.norm(g, axis=1, keepdims=True))
    tx = rng.standard_normal((rows, lay.d_in, C))
    tw = rng.standard_normal((rows, lay.n_paths, C))
    tdz = rng.standard_normal((rows, lay.d_out, C))
    dev = [torch.from_numpy(np.ascontiguousarray(a)).to("cuda") for a in (tx, y, tw, tdz)]
    z = e3.tp_fwd_f64(plan, *dev[:3])
    tdx, tdy, tdw = e3.tp_bwd_f64(plan, *dev)
    torch.cuda.synchronize()
    terrs = dict(z=rel_l2(to_np(z), otp.tp(lay, tx, y, tw).numpy()))
    for k, a, r in zip(("dx", "dy", "dw"), (tdx, tdy, tdw), otp.tp_bwd(lay, tx, y, tw, tdz)):
        terrs[k] = rel_l2(to_np(a), r.numpy())
    print("float64 tp rel-L2", terrs, flush=True)
    for k, v in terrs.items():
        assert v < TOL64, (k, v)


@pytest.mark.parametrize("irreps,lsh,lout,parity,n,e,K,pad", [
    ("16x0e+16x0o+16x1o+16x1e", 2, 2, "all", 50, 700, 8, 3),
    ("8x0o+8x1o", 1, 1, "natural", 40, 500, 5, -1),                 # a block with no path
    ("68x1o+68x2o", 3, 2, "all", 30, 400, 12, -1),                  # a ragged slab, K > 8
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, "all", 60, 1200, 8, 5),   # the benchmark layout, forced
])
def test_composed_radial(e3, irreps, lsh, lout, parity, n, e, K, pad):
    """The fused radial weights (s = h W on the matrix cores) on the composed
    path: m, dx, dvec, dh, dW against the oracle, bitwise repeats, zero
    cotangents of padding edges."""
    _say("composed radial", irreps, lsh, lout, parity, n, e, K, pad)
    rng = np.random.default_rng(49)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    plan = _plan(e3, irreps, lsh, lout, parity, "composed")
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
    h = rng.standard_normal((e, K)).astype(np.float32)
    W = (rng.standard_normal((K, lay.n_paths, C)) / np.sqrt(K)).astype(np.float32)
    dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    xs, vs, hs, Ws, dms = (to_dev(a) for a in (x, vec, h, W, dm))
    outs = []
    for _ in range(2):
        m = e3.conv_fwd_radial(plan, G, xs, vs, hs, Ws)
        outs.append([to_np(t) for t in (m,) + e3.conv_bwd_radial(plan, G, xs, vs, hs, Ws, dms)])
    for a, b in zip(*outs):
        assert np.array_equal(a, b), "not deterministic"
    m, dx, dvec, dh, dW = outs[0]
    ref_m = oradial.conv_fwd(lay, x, vec, h, W, snd, rcv, n, pad_node=pad).numpy()
    ref = oradial.conv_bwd(lay, x, vec, h, W, dm, snd, rcv, n, pad_node=pad)
    errs = dict(m=rel_l2(m, ref_m), dx=rel_l2(dx, ref["dx"].numpy()), dvec=rel_l2(dvec, ref["dvec"].numpy()),
                dh=rel_l2(dh, ref["dh"].numpy()), dW=rel_l2(dW, ref["dW"].numpy()))
    print("rel-L2", errs, flush=True)
    for k, v in errs.items():
        assert v < TOL, (k, v)
    if pad >= 0:
        dead = (snd == pad) | (rcv == pad)
        assert np.all(dh[dead] == 0) and np.all(dvec[dead] == 0)
        assert np.all(m[pad] == 0) and np.all(dx[pad] == 0)


def _random_layout(rng):
    """A random channelwise layout: 1-5 blocks of degree <= 3 with random
    parities, harmonics and outputs to degree 3, all or natural paths, C a
    multiple of 4 (re-drawn until it has a path)."""
    while True:
        nb = int(rng.integers(1, 6))
        C = 4 * int(rng.integers(1, 50))
        blocks = [f"{C}x{int(rng.integers(0, 4))}{'eo'[int(rng.integers(0, 2))]}" for _ in range(nb)]
        irreps = "+".join(blocks)
        lsh, lout = int(rng.integers(0, 4)), int(rng.integers(0, 4))
        parity = "natural" if rng.random() < 0.4 else "all"
        lay = oirreps.layout(irreps, lsh, lout, parity=parity)
        if lay.n_paths > 0:
            return irreps, lsh, lout, parity, lay


@pytest.mark.parametrize("seed", range(12))
def test_generic_random_layouts(e3, seed):
    """Seeded random layouts: the convolution forward and backward and the
    tensor product forward and backward on the composed path (and, for even
    seeds, the record path) against the oracle."""
    rng = np.random.default_rng(1000 + seed)
    irreps, lsh, lout, parity, lay = _random_layout(rng)
    n, e = int(rng.integers(10, 50)), int(rng.integers(50, 400))
    pad = int(rng.integers(0, n)) if seed % 3 == 0 else -1
    C = lay.channels
    snd, rcv, vec = _random_graph(rng, n, e)
    x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
    s = rng.standard_normal((e, lay.n_paths, C)).astype(np.float32)
    dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
    rows = int(rng.integers(1, 40))
    g = rng.standard_normal((rows, 3))
    y = osh.sh_unit(lsh, g / np.linalg.norm(g, axis=1, keepdims=True)).astype(np.float32)
    tx = rng.standard_normal((rows, lay.d_in, C)).astype(np.float32)
    tw = rng.standard_normal((rows, lay.n_paths, C)).astype(np.float32)
    tdz = rng.standard_normal((rows, lay.d_out, C)).astype(np.float32)
    ref_m = oconv.conv_fwd(lay, x, vec, s, snd, rcv, n, pad_node=pad).numpy()
    ref = oconv.conv_bwd(lay, x, vec, s, dm, snd, rcv, n, pad_node=pad)
    ref_z = otp.tp(lay, tx, y, tw).numpy()
    ref_t = otp.tp_bwd(lay, tx, y, tw, tdz)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
    for path in (("composed", "records") if seed % 2 == 0 else ("composed",)):
        _say("random layout", seed, path, irreps, lsh, lout, parity, n, e, pad, rows)
        plan = _plan(e3, irreps, lsh, lout, parity, path)
        xs, vs, ss, dms = to_dev(x), to_dev(vec), to_dev(s), to_dev(dm)
        m = e3.conv_fwd(plan, G, xs, vs, ss)
        dx, dvec, ds = e3.conv_bwd(plan, G, xs, vs, ss, dms)
        z = e3.tp_fwd(plan, to_dev(tx), to_dev(y), to_dev(tw))
        tdx, tdy, tdw = e3.tp_bwd(plan, to_dev(tx), to_dev(y), to_dev(tw), to_dev(tdz))
        errs = dict(m=rel_l2(to_np(m), ref_m), dx=rel_l2(to_np(dx), ref["dx"].numpy()),
                    ds=rel_l2(to_np(ds), ref["ds"].numpy()), dvec=rel_l2(to_np(dvec), ref["dvec"].numpy()),
                    z=rel_l2(to_np(z), ref_z), tdx=rel_l2(to_np(tdx), ref_t[0].numpy()),
                    tdy=rel_l2(to_np(tdy), ref_t[1].numpy()), tdw=rel_l2(to_np(tdw), ref_t[2].numpy()))
        print("rel-L2", errs, flush=True)
        for k, v in errs.items():
            assert v < TOL, (path, k, v)


@pytest.mark.parametrize("irreps,lsh,lout,parity", [
    ("16x0e+16x1o", 2, 2, "all"), ("16x0e+16x1o+16x2e", 2, 2, "all"), ("16x0e+16x1o", 3, 3, "all"),
    ("16x0e+16x1o+16x2e", 3, 3, "all"), ("16x0e+16x1o+16x2e+16x3o", 3, 3, "all"),
    ("16x0e+16x1o", 2, 2, "natural"), ("16x0e+16x1o", 3, 3, "natural"), ("16x0e+16x1o+16x2e", 3, 3, "natural"),
    ("16x0e+16x1o+16x2e+16x3o", 3, 3, "natural"), ("16x1o+16x0e+16x3o+16x2e", 3, 3, "all"),
])
def test_composed_equals_compiled_on_every_compiled_layout(e3, irreps, lsh, lout, parity):
    """Every compiled layout forced onto the composed path: convolution forward,
    backward and double backward, and the tensor product forward and backward,
    agree with the compiled kernels to float32 rounding (the two sum in
    different orders)."""
    import torch
    _say("composed vs compiled", irreps, lsh, lout, parity)
    rng = np.random.default_rng(50)
    lay = oirreps.layout(irreps, lsh, lout, parity=parity)
    nat = parity == "natural"
    cp = e3.Plan(irreps, lsh, lout, natural=nat)
    kp = e3.Plan(irreps, lsh, lout, natural=nat, composed=True)
    assert (cp.kernels, kp.kernels) == ("compiled", "composed")
    n, e, R = 40, 500, 33
    snd, rcv, vec = _random_graph(rng, n, e)
    C = lay.channels
    f = lambda *shape: to_dev(rng.standard_normal(shape).astype(np.float32))
    x, vs, s, dm = f(n, lay.d_in, C), to_dev(vec), f(e, lay.n_paths, C), f(n, lay.d_out, C)
    y, ddx, ddy, dds = f(e, lay.d_sh), f(n, lay.d_in, C), f(e, lay.d_sh), f(e, lay.n_paths, C)
    tx, ty, tw, tdz = f(R, lay.d_in, C), f(R, lay.d_sh), f(R, lay.n_paths, C), f(R, lay.d_out, C)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=3)

    def run(plan):
        out = [e3.conv_fwd(plan, G, x, vs, s)]
        out += list(e3.conv_bwd(plan, G, x, vs, s, dm))
        out += list(e3.conv_bwd2(plan, G, x, y, s, dm, ddx, ddy, dds))
        out += [e3.tp_fwd(plan, tx, ty, tw)]
        out += list(e3.tp_bwd(plan, tx, ty, tw, tdz))
        torch.cuda.synchronize()
        return out

    names = ["m", "dx", "dvec", "ds", "gx", "gy", "gs", "gdm", "z", "tdx", "tdy", "tdw"]
    for name, a, b in zip(names, run(kp), run(cp)):
        err = rel_l2(to_np(a), to_np(b))
        assert err < 1e-6, (name, err)
