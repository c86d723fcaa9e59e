"""The no-allocation backward (e3_conv_bwd_noalloc), called through the C ABI:
its outputs equal those of the workspace entry point (e3_conv_bwd) bit for bit
and the fp64 oracle to the parity bar, on two calls in a row, the second on a
smaller graph; a graph whose scratch exceeds the fixed array is refused; and a
captured call replays to the eager result.
"""
import numpy as np
import pytest

from gpu_util import TOL, rel_l2, to_dev, to_np
from oracle import conv as oconv
from oracle import irreps as oirreps

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def e3():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    from paper_2609_35099_amd import e3mi
    e3mi.lib()
    return e3mi


def _graph(rng, n, e, pad=-1):
    snd = rng.integers(0, n, e).astype(np.int32)
    rcv = rng.integers(0, n, e).astype(np.int32)
    rcv = np.where(rcv == snd, (rcv + 1) % n, rcv).astype(np.int32)
    vec = (rng.standard_normal((e, 3)) * 2.0).astype(np.float32)
    return snd, rcv, vec


@pytest.mark.parametrize("irreps,lsh,lout,force,kernels", [
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, False, "compiled"),
    ("64x1o+64x0e+64x1e", 2, 2, False, "composed"),                 # a layout without compiled kernels
    ("128x0e+128x1o+128x2e+128x3o", 3, 3, True, "composed"),        # forced onto the composed path
])
def test_noalloc_backward_equals_workspace_backward(e3, irreps, lsh, lout, force, kernels):
    import torch
    lay = oirreps.layout(irreps, lsh, lout)
    plan = e3.Plan(irreps, lsh, lout, composed=force)
    assert plan.kernels == kernels
    C = lay.channels
    rng = np.random.default_rng(74)
    # the second call is smaller, so it leaves the first call's partials in the
    # part of the scratch it does not use
    for n, e, pad in [(600, 7000, -1), (120, 1500, 5)]:
        print(f"[case] no-allocation backward, {irreps} {kernels} n={n} e={e} pad={pad}", flush=True)
        snd, rcv, vec = _graph(rng, n, e)
        if pad >= 0:
            snd[::97] = pad
        G = e3.Graph(to_dev(snd), to_dev(rcv), n, pad_node=pad)
        x = rng.standard_normal((n, lay.d_in, C)).astype(np.float32)
        s = rng.standard_normal((e, lay.n_paths, C)).astype(np.float32)
        dm = rng.standard_normal((n, lay.d_out, C)).astype(np.float32)
        xs, vs, ss, dms = to_dev(x), to_dev(vec), to_dev(s), to_dev(dm)
        assert e3.conv_workspace_size(plan, G)[1] <= e3.NOALLOC_SCRATCH_BYTES
        ref = e3.conv_bwd(plan, G, xs, vs, ss, dms)
        dx = torch.full((n, lay.d_in, C), float("nan"), device="cuda")
        dvec = torch.full((e, 3), float("nan"), device="cuda")
        ds = torch.full((e, lay.n_paths, C), float("nan"), device="cuda")
        e3.conv_bwd_noalloc(plan, G, xs, vs, ss, dms, dx, dvec, ds)
        torch.cuda.synchronize()
        for a, b in zip((dx, dvec, ds), ref):
            assert torch.equal(a, b)
        o = oconv.conv_bwd(lay, x, vec, s, dm, snd, rcv, n, pad_node=pad)
        errs = dict(dx=rel_l2(to_np(dx), o["dx"].numpy()), ds=rel_l2(to_np(ds), o["ds"].numpy()),
                    dvec=rel_l2(to_np(dvec), o["dvec"].numpy()))
        print("rel-L2", errs, flush=True)
        for k, v in errs.items():
            assert v < TOL, (k, v)


def test_noalloc_backward_refuses_a_graph_beyond_its_scratch(e3):
    import torch
    irreps = "128x0e+128x1o+128x2e+128x3o"
    lay = oirreps.layout(irreps, 3, 3)
    plan = e3.Plan(irreps, 3, 3)
    rng = np.random.default_rng(75)
    n, e = 2000, 9000
    snd, rcv, vec = _graph(rng, n, e)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n)
    assert e3.conv_workspace_size(plan, G)[1] > e3.NOALLOC_SCRATCH_BYTES
    C = lay.channels
    xs = torch.zeros((n, lay.d_in, C), device="cuda")
    dms = torch.zeros((n, lay.d_out, C), device="cuda")
    ss = torch.zeros((e, lay.n_paths, C), device="cuda")
    with pytest.raises(e3.E3Error) as ei:
        e3.conv_bwd_noalloc(plan, G, xs, to_dev(vec), ss, dms, torch.empty_like(xs),
                            torch.empty((e, 3), device="cuda"), torch.empty_like(ss))
    assert ei.value.status == 4


def test_noalloc_backward_in_captured_graph(e3):
    """The callers it is for: captured in a HIP graph with preallocated outputs
    (no workspace), every replay equals the eager call bit for bit, with eager
    work on the same scratch between replays."""
    import torch
    irreps = "128x0e+128x1o+128x2e+128x3o"
    lay = oirreps.layout(irreps, 3, 3)
    plan = e3.Plan(irreps, 3, 3)
    C = lay.channels
    rng = np.random.default_rng(76)
    n, e = 300, 4000
    print(f"[case] no-allocation backward in a captured graph, n={n} e={e}", flush=True)
    snd, rcv, vec = _graph(rng, n, e)
    G = e3.Graph(to_dev(snd), to_dev(rcv), n)
    xs = to_dev(rng.standard_normal((n, lay.d_in, C)).astype(np.float32))
    ss = to_dev(rng.standard_normal((e, lay.n_paths, C)).astype(np.float32))
    dms = to_dev(rng.standard_normal((n, lay.d_out, C)).astype(np.float32))
    vs = to_dev(vec)
    dx, dvec, ds = torch.empty_like(xs), torch.empty((e, 3), device="cuda"), torch.empty_like(ss)
    e3.conv_bwd_noalloc(plan, G, xs, vs, ss, dms, dx, dvec, ds)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (dx, dvec, ds)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        e3.conv_bwd_noalloc(plan, G, xs, vs, ss, dms, dx, dvec, ds)
    torch.cuda.synchronize()
    # another call on a smaller graph between replays overwrites part of the scratch
    m = 100
    G2 = e3.Graph(to_dev(snd[:1000] % m), to_dev(rcv[:1000] % m), m)
    x2, dm2 = xs[:m].contiguous(), dms[:m].contiguous()
    for it in range(3):
        for t in (dx, dvec, ds):
            t.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip((dx, dvec, ds), ref):
            assert torch.equal(a, b), it
        e3.conv_bwd_noalloc(plan, G2, x2, vs[:1000].contiguous(), ss[:1000].contiguous(), dm2,
                            torch.empty_like(x2), torch.empty((1000, 3), device="cuda"),
                            torch.empty((1000, lay.n_paths, C), device="cuda"))
        torch.cuda.synchronize()
