"""CPU-side checks of the HIP library: it loads, exports every symbol the
header declares, validates arguments, and its host-built tables (the
ladder-operator Clebsch-Gordan construction and the harmonic polynomials)
equal the oracle's independent ones.  No device work is launched here.
"""
import ctypes as ct
import os
import re

import numpy as np
import pytest

from oracle import cg as ocg
from oracle import irreps as oirreps
from oracle import sh as osh
from paper_2609_35099_amd import e3mi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "e3mi.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(e3_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = e3mi.lib()
    names = _declared()
    assert len(names) >= 18
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(e3mi.SIGNATURES), "binding and header disagree"


def test_status_strings():
    L = e3mi.lib()
    for s in range(7):
        assert L.e3_status_str(s)


LAYOUTS = [("8x0e+8x1o", 2, 2), ("128x0e+128x1o+128x2e", 3, 3), ("128x0e+128x1o", 3, 3),
           ("128x0e+128x1o+128x2e+128x3o", 3, 3), ("64x0e+64x1o+64x2e+64x3o", 3, 3),
           ("4x1o+4x0e+4x2o", 2, 3)]


@pytest.mark.parametrize("natural", [False, True])
@pytest.mark.parametrize("spec", LAYOUTS + [("4x0o+4x1e", 2, 2), ("128x1o+128x0e+128x3o+128x2e", 3, 3)])
def test_plan_tables_equal_oracle(spec, natural):
    plan = e3mi.Plan(*spec, natural=natural)
    lay = oirreps.layout(*spec, parity="natural" if natural else "all")
    assert (plan.P, plan.D_in, plan.D_sh, plan.D_out, plan.C) == \
        (lay.n_paths, lay.d_in, lay.d_sh, lay.d_out, lay.channels)
    paths = plan.paths()
    for row, p in zip(paths, lay.paths):
        assert tuple(row) == (p.l1, p.l2, p.l3, p.p3, p.x_off, p.y_off, p.out_off)
    i0, i1, i2, v = plan.records()
    ref = ocg.coo_records(lay)
    assert len(ref) == len(v) == plan.info.nnz
    assert [(a, b, c) for a, b, c, _ in ref] == list(zip(i0.tolist(), i1.tolist(), i2.tolist()))
    assert np.abs(np.array([r[3] for r in ref]) - v).max() < 1e-12


def test_plan_supported_variants():
    for spec in LAYOUTS[:5]:
        assert e3mi.Plan(*spec).kernels == "compiled", spec
        assert e3mi.Plan(*spec, natural=True).kernels == "compiled", spec
    # any parities select the same kernels when every path is kept; a reordered
    # block list has its own compiled kernels
    assert e3mi.Plan("128x0o+128x1e+128x2o+128x3e", 3, 3).kernels == "compiled"
    assert e3mi.Plan("128x1o+128x0e+128x3o+128x2e", 3, 3).kernels == "compiled"
    # natural parities of other x parities select other paths: not compiled
    assert e3mi.Plan("128x0o+128x1e", 2, 2, natural=True).kernels != "compiled"


def test_plan_without_kernels_is_valid_and_refuses_compute():
    """A layout neither the composed nor the record path takes (an x block of
    degree 4) is still a plan with queryable tables; its compute calls report
    E3_ERR_UNSUPPORTED.  Any layout of degrees <= 3 is composed of
    single-block kinds (no device tables needed)."""
    p = e3mi.Plan("4x1o+4x0e+4x4o", 2, 3)
    assert not p.supported and p.kernels is None and p.info.nnz > 0
    with pytest.raises(e3mi.E3Error) as ei:
        st = e3mi.lib().e3_tp_fwd(p.handle, None, None, None, None, 1, None)
        e3mi._check(st, "e3_tp_fwd")
    assert ei.value.status == 2
    q = e3mi.Plan("4x1o+4x0e+4x2o", 2, 3)
    assert q.kernels == "composed"


@pytest.mark.parametrize("spec", [("16x0e+16x0o+16x1o+16x1e", 2, 2, False), ("32x2e+32x0e+32x1o", 3, 3, False),
                                  ("8x3o+8x1e", 1, 3, True), ("68x1o+68x2o", 3, 2, False), ("4x0e", 0, 0, False),
                                  ("8x0o+8x1o", 1, 1, True), ("1024x1o+1024x1e", 1, 1, False),
                                  ("64x0e+64x1o+64x1e+64x2e+64x3o", 3, 3, True),
                                  ("4x0e+4x1o+4x2e+4x3o+4x0o+4x1e+4x2o+4x3e", 3, 3, False)])
def test_record_tables_pass_their_bounds_check(spec):
    """The record path's tables of layouts without compiled kernels are built
    and pass the bounds check of every index the kernels read, before the
    device upload: here, without a device, creation stops only at the upload.
    Without the flag, the same layouts are composed of single-block kinds."""
    irreps, lsh, lout, natural = spec
    assert e3mi.Plan(irreps, lsh, lout, natural=natural).kernels == "composed"
    p = e3mi.Plan(irreps, lsh, lout, natural=natural, records=True)
    if p.kernels == "records":
        return
    assert p.kernels is None
    with pytest.raises(e3mi.E3Error) as ei:
        e3mi._check(e3mi.lib().e3_tp_fwd(p.handle, None, None, None, None, 1, None), "e3_tp_fwd")
    assert ei.value.status == 2 and "no device" in str(ei.value), str(ei.value)


def test_record_path_refuses_degree_4_and_unknown_flags():
    p = e3mi.Plan("4x0e+4x4o", 2, 3)
    with pytest.raises(e3mi.E3Error) as ei:
        e3mi._check(e3mi.lib().e3_tp_fwd(p.handle, None, None, None, None, 1, None), "e3_tp_fwd")
    assert ei.value.status == 2 and "degree up to 3" in str(ei.value), str(ei.value)
    h = ct.c_void_p()
    assert e3mi.lib().e3_plan_create(b"4x0e", 0, 0, 8, ct.byref(h)) == 1    # unknown flag
    assert e3mi.lib().e3_plan_create(b"4x0e", 0, 0, 2 | 4, ct.byref(h)) == 1  # records and composed
    c = e3mi.Plan("4x0e+4x4o", 2, 3, composed=True)
    assert c.kernels is None
    with pytest.raises(e3mi.E3Error) as ei:
        e3mi._check(e3mi.lib().e3_tp_fwd(c.handle, None, None, None, None, 1, None), "e3_tp_fwd")
    assert ei.value.status == 2 and "composed path" in str(ei.value), str(ei.value)
    # a compiled layout forced onto the composed path
    assert e3mi.Plan("128x0e+128x1o+128x2e+128x3o", 3, 3, composed=True).kernels == "composed"


def test_natural_parity_filter():
    p = e3mi.Plan("4x0e+4x1o", 2, 2, natural=True)
    lay = oirreps.layout("4x0e+4x1o", 2, 2, parity="natural")
    assert p.P == lay.n_paths < oirreps.layout("4x0e+4x1o", 2, 2).n_paths


def test_sh_host_equals_oracle():
    rng = np.random.default_rng(0)
    g = rng.standard_normal((100, 3))
    u = g / np.linalg.norm(g, axis=1, keepdims=True)
    for l in range(4):
        assert np.abs(e3mi.sh_host(l, u) - osh.sh_unit(l, u)).max() < 1e-13


@pytest.mark.parametrize("args", [("", 2, 2), ("8x0e+4x1o", 2, 2), ("8x0q", 2, 2), ("8x0e", -1, 2),
                                  ("8x0e", 4, 2), ("x0e", 2, 2), ("8x0e++8x1o", 2, 2)])
def test_plan_create_rejects_bad_input(args):
    with pytest.raises(e3mi.E3Error) as ei:
        e3mi.Plan(*args)
    assert ei.value.status in (1, 2)


def test_null_and_negative_arguments_rejected_before_device_work():
    L = e3mi.lib()
    h = ct.c_void_p()
    assert L.e3_plan_create(None, 2, 2, 0, ct.byref(h)) == 1
    assert L.e3_plan_create(b"8x0e", 2, 2, 7, ct.byref(h)) == 1
    assert L.e3_sh(5, None, None, 10, None) == 1
    assert L.e3_sh(2, None, None, -1, None) == 1
    assert L.e3_sh(2, None, None, 0, None) == 0          # empty input is a no-op
    assert L.e3_sh_bwd(2, None, None, None, 3, None) == 1
    assert L.e3_sh_host(2, None, None, 3) == 1
    assert L.e3_graph_create(None, None, 10, 5, -1, None, ct.byref(h)) == 1
    assert L.e3_graph_create(None, None, -1, 0, -1, None, ct.byref(h)) == 1
    assert L.e3_graph_create(None, None, 10, 0, 12, None, ct.byref(h)) == 1
    assert L.e3_conv_fwd(None, None, None, None, None, None, None, 0, None) == 1
    assert L.e3_conv_bwd(None, None, None, None, None, None, None, None, None, None, 0, None) == 1
    plan = e3mi.Plan("8x0e+8x1o", 2, 2)
    assert L.e3_conv_fwd(plan.handle, None, None, None, None, None, None, 0, None) == 1
    assert L.e3_tp_fwd(plan.handle, None, None, None, None, -1, None) == 1
    assert L.e3_tp_fwd(plan.handle, None, None, None, None, 0, None) == 0
    assert L.e3_tp_fwd(plan.handle, None, None, None, None, 4, None) == 1
    # misaligned pointers are refused
    assert L.e3_tp_fwd(plan.handle, ct.c_void_p(4), ct.c_void_p(4), ct.c_void_p(4), ct.c_void_p(4), 4, None) == 1
    # tensor product backward: argument checks and workspace sizing, no device work
    n = ct.c_size_t()
    assert L.e3_tp_workspace_size(plan.handle, -1, ct.byref(n)) == 1
    assert L.e3_tp_workspace_size(plan.handle, 10, None) == 1
    assert L.e3_tp_workspace_size(plan.handle, 10, ct.byref(n)) == 0 and n.value >= 10 * 16 * 4
    assert n.value % 256 == 0
    nul = [None] * 7
    assert L.e3_tp_bwd(plan.handle, *nul, None, 0, -1, None) == 1
    assert L.e3_tp_bwd(plan.handle, *nul, None, 0, 0, None) == 0
    assert L.e3_tp_bwd(plan.handle, *nul, None, 0, 3, None) == 1
    fake = [ct.c_void_p(256)] * 7
    assert L.e3_tp_bwd(plan.handle, *fake, ct.c_void_p(256), 16, 10, None) == 4   # workspace too small
    assert L.e3_tp_bwd(plan.handle, *([ct.c_void_p(4)] * 7), ct.c_void_p(256), n.value, 10, None) == 1
    # fused radial weights: a graph is required, K must lie in [1, 16]
    assert L.e3_conv_radial_workspace_size(plan.handle, None, 8, ct.byref(n)) == 1
    assert L.e3_conv_fwd_radial(plan.handle, None, None, None, None, None, 8, None, None) == 1
    assert L.e3_conv_bwd_radial(plan.handle, None, None, None, None, None, 8, None, None, None, None, None,
                                None, 0, None) == 1
    assert L.e3_conv_fwd_radial(None, None, None, None, None, None, 8, None, None) == 1


def test_linear_descriptor_rejects_bad_layouts():
    """Linear-mixing descriptor: layouts it cannot take are refused before any
    device work (host only; valid descriptors upload their tables to the
    current device, so they are checked by the GPU tests)."""
    for bad in [("8x0e", "16x0e"), ("16x0e+8x1o", "16x0e"), ("", "16x0e")]:
        with pytest.raises(e3mi.E3Error) as ei:
            e3mi.Linear(*bad)
        assert ei.value.status in (1, 2)


def test_record_tp_create_checks():
    """Record tensor product descriptor: index, size and staging-limit checks,
    all made before the tables are uploaded (host only)."""
    L = e3mi.lib()
    h = ct.c_void_p()
    i = (ct.c_int32 * 2)(0, 1)
    v = (ct.c_double * 2)(1.0, 2.0)
    bad = (ct.c_int32 * 2)(0, 4)
    assert L.e3_tpg_create(4, 4, 4, 2, bad, i, i, v, 1, ct.byref(h)) == 3
    assert L.e3_tpg_create(0, 4, 4, 2, i, i, i, v, 1, ct.byref(h)) == 1
    assert L.e3_tpg_create(4, 4, 4, 2, None, i, i, v, 1, ct.byref(h)) == 1
    assert L.e3_tpg_create(4, 4, 400, 2, i, i, i, v, 1, ct.byref(h)) == 2     # 400 rows x 64 lanes > 64 KiB
    assert L.e3_tpg_create(4, 4, 4, 2, i, i, i, v, 1, None) == 1


def test_probe_stream_argument_checks():
    """Streaming probe: argument and shape checks, all before device work."""
    L = e3mi.lib()
    br, bw = ct.c_size_t(), ct.c_size_t()
    fake = ct.c_void_p(256)
    assert L.e3_probe_stream(fake, 1024, fake, 1024, 0, 0, 16, 0, ct.byref(br), ct.byref(bw), None) == 1
    assert L.e3_probe_stream(fake, 1024, fake, 1024, 16, 0, 12, 0, ct.byref(br), ct.byref(bw), None) == 1
    assert L.e3_probe_stream(fake, 1024, fake, 1024, 16, 0, 16, 4, ct.byref(br), ct.byref(bw), None) == 1
    assert L.e3_probe_stream(None, 1024, fake, 1024, 16, 0, 16, 0, ct.byref(br), ct.byref(bw), None) == 1
    assert L.e3_probe_stream(ct.c_void_p(4), 1024, fake, 1024, 16, 0, 16, 0, ct.byref(br), ct.byref(bw),
                             None) == 1
    assert L.e3_probe_stream(fake, 1024, fake, 1024, 16, 0, 16, 0, None, ct.byref(bw), None) == 1
    # a read:write shape that is not compiled
    assert L.e3_probe_stream(fake, 1024, fake, 1024, 3, 5, 4, 0, ct.byref(br), ct.byref(bw), None) == 2
