"""Python binding of libe3mi (ctypes): argument marshalling only.

Every computation runs in the HIP library; this module checks tensor shapes,
dtypes and devices, passes raw device pointers and the current torch stream,
and raises E3Error on a non-OK status.  If the library has not been built the
first call raises (there is no fallback path).
"""
from __future__ import annotations

import ctypes as ct
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# E3MI_LIB may point at another build of the same library (side-by-side builds)
LIB_PATH = os.environ.get("E3MI_LIB") or os.path.join(_HERE, "libe3mi.so")

_STATUS = {0: "E3_OK", 1: "E3_ERR_INVALID_ARG", 2: "E3_ERR_UNSUPPORTED",
           3: "E3_ERR_INDEX_OUT_OF_RANGE", 4: "E3_ERR_WORKSPACE_TOO_SMALL",
           5: "E3_ERR_HIP", 6: "E3_ERR_ALLOC"}

E3_PARITY_ALL = 0
E3_PARITY_NATURAL = 1
E3_PLAN_RECORDS = 2
E3_PLAN_COMPOSED = 4


class E3Error(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        name = _STATUS.get(status, str(status))
        super().__init__(f"{where}: {name}" + (f" ({detail})" if detail else ""))


class PlanInfo(ct.Structure):
    _fields_ = [("C", ct.c_int), ("P", ct.c_int), ("D_in", ct.c_int), ("D_sh", ct.c_int),
                ("D_out", ct.c_int), ("nnz", ct.c_int), ("lmax_sh", ct.c_int),
                ("lmax_out", ct.c_int), ("supported", ct.c_int)]


_lib = None

# name -> (restype, argtypes); mirrors include/e3mi.h
_P, _I, _I64, _U, _D = ct.c_void_p, ct.c_int, ct.c_int64, ct.c_uint, ct.c_double
SIGNATURES = {
    "e3_plan_create": (_I, [ct.c_char_p, _I, _I, _U, ct.POINTER(_P)]),
    "e3_plan_query": (_I, [_P, ct.POINTER(PlanInfo)]),
    "e3_plan_destroy": (_I, [_P]),
    "e3_plan_paths": (_I, [_P, _P]),
    "e3_plan_records": (_I, [_P, _I64, _P, _P, _P, _P, ct.POINTER(_I64)]),
    "e3_sh_host": (_I, [_I, _P, _P, _I64]),
    "e3_graph_create": (_I, [_P, _P, _I64, _I64, ct.c_int32, _P, ct.POINTER(_P)]),
    "e3_graph_live_edges": (_I, [_P, ct.POINTER(_I64)]),
    "e3_graph_export": (_I, [_P, _P, _P, _P, _P]),
    "e3_graph_destroy": (_I, [_P]),
    "e3_sh": (_I, [_I, _P, _P, _I64, _P]),
    "e3_sh_bwd": (_I, [_I, _P, _P, _P, _I64, _P]),
    "e3_tp_fwd": (_I, [_P, _P, _P, _P, _P, _I64, _P]),
    "e3_tp_workspace_size": (_I, [_P, _I64, ct.POINTER(ct.c_size_t)]),
    "e3_tp_bwd": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _I64, _P]),
    "e3_conv_workspace_size": (_I, [_P, _P, ct.POINTER(ct.c_size_t), ct.POINTER(ct.c_size_t)]),
    "e3_linear_create": (_I, [ct.c_char_p, ct.c_char_p, ct.POINTER(ct.c_void_p)]),
    "e3_linear_query": (_I, [_P, ct.POINTER(ct.c_int64), ct.POINTER(ct.c_int), ct.POINTER(ct.c_int),
                             ct.POINTER(ct.c_int), ct.POINTER(ct.c_int)]),
    "e3_linear_destroy": (_I, [_P]),
    "e3_linear_fwd": (_I, [_P, _P, _P, _P, _I64, _P]),
    "e3_linear_workspace_size": (_I, [_P, ct.POINTER(ct.c_size_t)]),
    "e3_linear_bwd": (_I, [_P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _I64, _P]),
    "e3_tpg_create": (_I, [ct.c_int, ct.c_int, ct.c_int, _I64, _P, _P, _P, _P, ct.c_int, ct.POINTER(ct.c_void_p)]),
    "e3_tpg_destroy": (_I, [_P]),
    "e3_tpg_fwd": (_I, [_P, _P, _P, _P, _I64, ct.c_int, _P]),
    "e3_tpg_workspace_size": (_I, [_P, _I64, ct.c_int, ct.POINTER(ct.c_size_t)]),
    "e3_tpg_bwd": (_I, [_P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _I64, ct.c_int, _P]),
    "e3_tpg_fwd_f64": (_I, [_P, _P, _P, _P, _I64, ct.c_int, _P]),
    "e3_tpg_bwd_f64": (_I, [_P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _I64, ct.c_int, _P]),
    "e3_conv_fwd_y": (_I, [_P, _P, _P, _P, _P, _P, ct.c_int, _P]),
    "e3_conv_bwd_y": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, ct.c_int, _P, ct.c_size_t, _P]),
    "e3_conv_bwd2": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _P]),
    "e3_conv_radial_workspace_size": (_I, [_P, _P, ct.c_int, ct.POINTER(ct.c_size_t)]),
    "e3_conv_fwd_radial": (_I, [_P, _P, _P, _P, _P, _P, ct.c_int, _P, _P]),
    "e3_conv_bwd_radial": (_I, [_P, _P, _P, _P, _P, _P, ct.c_int, _P, _P, _P, _P, _P, _P, ct.c_size_t, _P]),
    "e3_conv_fwd": (_I, [_P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _P]),
    "e3_conv_bwd": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _P]),
    "e3_conv_bwd_noalloc": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "e3_tp_fwd_f64": (_I, [_P, _P, _P, _P, _P, _I64, _P]),
    "e3_tp_workspace_size_f64": (_I, [_P, _I64, ct.POINTER(ct.c_size_t)]),
    "e3_tp_bwd_f64": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _I64, _P]),
    "e3_conv_workspace_size_f64": (_I, [_P, _P, ct.POINTER(ct.c_size_t)]),
    "e3_conv_fwd_f64": (_I, [_P, _P, _P, _P, _P, _P, _P]),
    "e3_conv_bwd_f64": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ct.c_size_t, _P]),
    "e3_probe_stream": (_I, [_P, ct.c_size_t, _P, ct.c_size_t, _I, _I, _I, _U, ct.POINTER(ct.c_size_t),
                             ct.POINTER(ct.c_size_t), _P]),
    "e3_timing_enable": (_I, [_I]),
    "e3_timing_reset": (_I, []),
    "e3_timing_read": (_I, [_I, _P, _P, _P, ct.POINTER(_I)]),
    "e3_status_str": (ct.c_char_p, [_I]),
    "e3_last_error": (ct.c_char_p, []),
}


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ct.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status: int, where: str):
    if status != 0:
        detail = lib().e3_last_error().decode(errors="replace")
        raise E3Error(status, where, detail)


# ---------------------------------------------------------------- tensors
def _torch():
    import torch
    return torch


def _ptr(t, name, shape=None, dtype="float32"):
    torch = _torch()
    want = {"float32": torch.float32, "float64": torch.float64, "int32": torch.int32}[dtype]
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype != want:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return ct.c_void_p(t.data_ptr()) if t.numel() else ct.c_void_p(0)


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ct.c_void_p(s.cuda_stream)


def _on_stream(fn):
    """Run a compute call with the caller's stream made current, so that the
    outputs and the workspace it allocates belong to that stream in torch's
    caching allocator (their memory is not handed out again while the kernels
    launched on that stream may still use it)."""
    import functools

    @functools.wraps(fn)
    def wrapped(*args, stream=None, **kw):
        if stream is None:
            return fn(*args, **kw)
        with _torch().cuda.stream(stream):
            return fn(*args, stream=stream, **kw)
    return wrapped


# ---------------------------------------------------------------- plan
class Plan:
    """Paths, coupling tables and kernels for an irreps layout.

    `kernels` is "compiled" when a kernel variant was generated for the layout,
    "composed" when it runs block by block on generated single-block kernels,
    "records" when it runs on the record path (its coupling records uploaded
    to the current device at creation), else None (no compute).
    """

    def __init__(self, irreps: str, lmax_sh: int, lmax_out: int, natural: bool = False,
                 records: bool = False, composed: bool = False):
        h = ct.c_void_p()
        flags = ((E3_PARITY_NATURAL if natural else E3_PARITY_ALL) | (E3_PLAN_RECORDS if records else 0)
                 | (E3_PLAN_COMPOSED if composed else 0))
        _check(lib().e3_plan_create(irreps.encode(), lmax_sh, lmax_out, flags, ct.byref(h)),
               "e3_plan_create")
        self._h = h
        info = PlanInfo()
        _check(lib().e3_plan_query(h, ct.byref(info)), "e3_plan_query")
        self.info = info
        self.irreps = irreps
        self.C, self.P = info.C, info.P
        self.D_in, self.D_sh, self.D_out = info.D_in, info.D_sh, info.D_out
        self.supported = bool(info.supported)
        self.kernels = {1: "compiled", 2: "records", 3: "composed"}.get(info.supported)

    @property
    def handle(self):
        return self._h

    def paths(self) -> np.ndarray:
        out = np.zeros((self.P, 7), dtype=np.int32)
        _check(lib().e3_plan_paths(self._h, out.ctypes.data_as(ct.c_void_p)), "e3_plan_paths")
        return out

    def records(self):
        n = ct.c_int64()
        _check(lib().e3_plan_records(self._h, 0, None, None, None, None, ct.byref(n)), "e3_plan_records")
        m = n.value
        i0, i1, i2 = (np.zeros(m, np.int32) for _ in range(3))
        v = np.zeros(m, np.float64)
        _check(lib().e3_plan_records(self._h, m, i0.ctypes.data_as(ct.c_void_p), i1.ctypes.data_as(ct.c_void_p),
                                     i2.ctypes.data_as(ct.c_void_p), v.ctypes.data_as(ct.c_void_p),
                                     ct.byref(n)), "e3_plan_records")
        return i0, i1, i2, v

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            lib().e3_plan_destroy(self._h)
            self._h = ct.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def sh_host(lmax: int, u: np.ndarray) -> np.ndarray:
    """The builder's harmonic polynomials evaluated on the host (float64)."""
    u = np.ascontiguousarray(u, dtype=np.float64)
    y = np.zeros((u.shape[0], (lmax + 1) ** 2))
    _check(lib().e3_sh_host(lmax, u.ctypes.data_as(ct.c_void_p), y.ctypes.data_as(ct.c_void_p), u.shape[0]),
           "e3_sh_host")
    return y


# ---------------------------------------------------------------- graph
class Graph:
    """Receiver- and sender-sorted CSR of an edge list, built on the device."""

    def __init__(self, sender, receiver, n_nodes: int, pad_node: int = -1, stream=None):
        E = sender.shape[0]
        ps = _ptr(sender, "sender", (E,), "int32")
        pr = _ptr(receiver, "receiver", (E,), "int32")
        h = ct.c_void_p()
        _check(lib().e3_graph_create(ps, pr, n_nodes, E, pad_node, _stream(stream), ct.byref(h)),
               "e3_graph_create")
        self._h = h
        self.n_nodes, self.n_edges, self.pad_node = n_nodes, E, pad_node
        n = ct.c_int64()
        _check(lib().e3_graph_live_edges(h, ct.byref(n)), "e3_graph_live_edges")
        self.n_live = n.value

    @property
    def handle(self):
        return self._h

    def export(self):
        torch = _torch()
        dev = torch.device("cuda")
        pr = torch.empty(self.n_live, dtype=torch.int32, device=dev)
        rr = torch.empty(self.n_nodes + 1, dtype=torch.int32, device=dev)
        ps = torch.empty(self.n_live, dtype=torch.int32, device=dev)
        rs = torch.empty(self.n_nodes + 1, dtype=torch.int32, device=dev)
        torch.cuda.synchronize()
        _check(lib().e3_graph_export(self._h, _ptr(pr, "perm_r", dtype="int32"), _ptr(rr, "rowptr_r", dtype="int32"),
                                     _ptr(ps, "perm_s", dtype="int32"), _ptr(rs, "rowptr_s", dtype="int32")),
               "e3_graph_export")
        return pr, rr, ps, rs

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            lib().e3_graph_destroy(self._h)
            self._h = ct.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- compute
def _empty(shape, like=None):
    torch = _torch()
    return torch.empty(shape, dtype=torch.float32, device="cuda")


@_on_stream
def sh(lmax: int, vec, out=None, stream=None):
    n = vec.shape[0]
    out = _empty((n, (lmax + 1) ** 2)) if out is None else out
    _check(lib().e3_sh(lmax, _ptr(vec, "vec", (n, 3)), _ptr(out, "y", (n, (lmax + 1) ** 2)), n, _stream(stream)),
           "e3_sh")
    return out


@_on_stream
def sh_bwd(lmax: int, vec, dy, out=None, stream=None):
    n = vec.shape[0]
    out = _empty((n, 3)) if out is None else out
    _check(lib().e3_sh_bwd(lmax, _ptr(vec, "vec", (n, 3)), _ptr(dy, "dy", (n, (lmax + 1) ** 2)),
                           _ptr(out, "dvec", (n, 3)), n, _stream(stream)), "e3_sh_bwd")
    return out


@_on_stream
def tp_fwd(plan: Plan, x, y, w, out=None, stream=None):
    R = x.shape[0]
    out = _empty((R, plan.D_out, plan.C)) if out is None else out
    _check(lib().e3_tp_fwd(plan.handle, _ptr(x, "x", (R, plan.D_in, plan.C)), _ptr(y, "y", (R, plan.D_sh)),
                           _ptr(w, "w", (R, plan.P, plan.C)), _ptr(out, "z", (R, plan.D_out, plan.C)), R,
                           _stream(stream)), "e3_tp_fwd")
    return out


def tp_workspace_size(plan: Plan, rows: int) -> int:
    b = ct.c_size_t()
    _check(lib().e3_tp_workspace_size(plan.handle, rows, ct.byref(b)), "e3_tp_workspace_size")
    return b.value


@_on_stream
def tp_bwd(plan: Plan, x, y, w, dz, dx=None, dy=None, dw=None, ws=None, stream=None):
    """(dx, dy, dw) of the weighted tensor product."""
    R = x.shape[0]
    dx = _empty((R, plan.D_in, plan.C)) if dx is None else dx
    dy = _empty((R, plan.D_sh)) if dy is None else dy
    dw = _empty((R, plan.P, plan.C)) if dw is None else dw
    if ws is None:
        ws = workspace(tp_workspace_size(plan, R))
    _check(lib().e3_tp_bwd(plan.handle, _ptr(x, "x", (R, plan.D_in, plan.C)), _ptr(y, "y", (R, plan.D_sh)),
                           _ptr(w, "w", (R, plan.P, plan.C)), _ptr(dz, "dz", (R, plan.D_out, plan.C)),
                           _ptr(dx, "dx", (R, plan.D_in, plan.C)), _ptr(dy, "dy", (R, plan.D_sh)),
                           _ptr(dw, "dw", (R, plan.P, plan.C)), ct.c_void_p(ws.data_ptr()), ws.numel(), R,
                           _stream(stream)), "e3_tp_bwd")
    return dx, dy, dw


def conv_workspace_size(plan: Plan, graph: Graph):
    f, b = ct.c_size_t(), ct.c_size_t()
    _check(lib().e3_conv_workspace_size(plan.handle, graph.handle, ct.byref(f), ct.byref(b)),
           "e3_conv_workspace_size")
    return f.value, b.value


def workspace(nbytes: int):
    torch = _torch()
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device="cuda")


@_on_stream
def conv_fwd(plan: Plan, graph: Graph, x, vec, s, out=None, stream=None):
    N, E = graph.n_nodes, graph.n_edges
    out = _empty((N, plan.D_out, plan.C)) if out is None else out
    _check(lib().e3_conv_fwd(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C)),
                             _ptr(vec, "vec", (E, 3)), _ptr(s, "s", (E, plan.P, plan.C)),
                             _ptr(out, "m", (N, plan.D_out, plan.C)), None, 0, _stream(stream)), "e3_conv_fwd")
    return out


@_on_stream
def conv_bwd(plan: Plan, graph: Graph, x, vec, s, dm, dx=None, dvec=None, ds=None, ws=None, stream=None):
    N, E = graph.n_nodes, graph.n_edges
    dx = _empty((N, plan.D_in, plan.C)) if dx is None else dx
    dvec = _empty((E, 3)) if dvec is None else dvec
    ds = _empty((E, plan.P, plan.C)) if ds is None else ds
    if ws is None:
        ws = workspace(conv_workspace_size(plan, graph)[1])
    _check(lib().e3_conv_bwd(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C)),
                             _ptr(vec, "vec", (E, 3)), _ptr(s, "s", (E, plan.P, plan.C)),
                             _ptr(dm, "dm", (N, plan.D_out, plan.C)), _ptr(dx, "dx", (N, plan.D_in, plan.C)),
                             _ptr(dvec, "dvec", (E, 3)), _ptr(ds, "ds", (E, plan.P, plan.C)),
                             ct.c_void_p(ws.data_ptr()), ws.numel(), _stream(stream)), "e3_conv_bwd")
    return dx, dvec, ds


# ---------------------------------------------------------------- float64 builds
def _empty64(shape):
    torch = _torch()
    return torch.empty(shape, dtype=torch.float64, device="cuda")


@_on_stream
def tp_fwd_f64(plan: Plan, x, y, w, out=None, stream=None):
    R = x.shape[0]
    out = _empty64((R, plan.D_out, plan.C)) if out is None else out
    f = "float64"
    _check(lib().e3_tp_fwd_f64(plan.handle, _ptr(x, "x", (R, plan.D_in, plan.C), f), _ptr(y, "y", (R, plan.D_sh), f),
                               _ptr(w, "w", (R, plan.P, plan.C), f), _ptr(out, "z", (R, plan.D_out, plan.C), f), R,
                               _stream(stream)), "e3_tp_fwd_f64")
    return out


@_on_stream
def tp_bwd_f64(plan: Plan, x, y, w, dz, stream=None):
    R = x.shape[0]
    f = "float64"
    dx, dy, dw = _empty64((R, plan.D_in, plan.C)), _empty64((R, plan.D_sh)), _empty64((R, plan.P, plan.C))
    b = ct.c_size_t()
    _check(lib().e3_tp_workspace_size_f64(plan.handle, R, ct.byref(b)), "e3_tp_workspace_size_f64")
    ws = workspace(b.value)
    _check(lib().e3_tp_bwd_f64(plan.handle, _ptr(x, "x", (R, plan.D_in, plan.C), f), _ptr(y, "y", (R, plan.D_sh), f),
                               _ptr(w, "w", (R, plan.P, plan.C), f), _ptr(dz, "dz", (R, plan.D_out, plan.C), f),
                               _ptr(dx, "dx", (R, plan.D_in, plan.C), f), _ptr(dy, "dy", (R, plan.D_sh), f),
                               _ptr(dw, "dw", (R, plan.P, plan.C), f), ct.c_void_p(ws.data_ptr()), ws.numel(), R,
                               _stream(stream)), "e3_tp_bwd_f64")
    return dx, dy, dw


@_on_stream
def conv_fwd_f64(plan: Plan, graph: Graph, x, vec, s, out=None, stream=None):
    N, E = graph.n_nodes, graph.n_edges
    f = "float64"
    out = _empty64((N, plan.D_out, plan.C)) if out is None else out
    _check(lib().e3_conv_fwd_f64(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C), f),
                                 _ptr(vec, "vec", (E, 3), f), _ptr(s, "s", (E, plan.P, plan.C), f),
                                 _ptr(out, "m", (N, plan.D_out, plan.C), f), _stream(stream)), "e3_conv_fwd_f64")
    return out


@_on_stream
def conv_bwd_f64(plan: Plan, graph: Graph, x, vec, s, dm, stream=None):
    N, E = graph.n_nodes, graph.n_edges
    f = "float64"
    dx, dvec, ds = _empty64((N, plan.D_in, plan.C)), _empty64((E, 3)), _empty64((E, plan.P, plan.C))
    b = ct.c_size_t()
    _check(lib().e3_conv_workspace_size_f64(plan.handle, graph.handle, ct.byref(b)), "e3_conv_workspace_size_f64")
    ws = workspace(b.value)
    _check(lib().e3_conv_bwd_f64(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C), f),
                                 _ptr(vec, "vec", (E, 3), f), _ptr(s, "s", (E, plan.P, plan.C), f),
                                 _ptr(dm, "dm", (N, plan.D_out, plan.C), f), _ptr(dx, "dx", (N, plan.D_in, plan.C), f),
                                 _ptr(dvec, "dvec", (E, 3), f), _ptr(ds, "ds", (E, plan.P, plan.C), f),
                                 ct.c_void_p(ws.data_ptr()), ws.numel(), _stream(stream)), "e3_conv_bwd_f64")
    return dx, dvec, ds


NOALLOC_SCRATCH_BYTES = 64 << 20


def conv_bwd_noalloc(plan: Plan, graph: Graph, x, vec, s, dm, dx, dvec, ds, stream=None):
    """conv_bwd into the caller's outputs with the library's fixed scratch
    (no allocation by the library or here; outputs must be given)."""
    N, E = graph.n_nodes, graph.n_edges
    _check(lib().e3_conv_bwd_noalloc(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C)),
                                     _ptr(vec, "vec", (E, 3)), _ptr(s, "s", (E, plan.P, plan.C)),
                                     _ptr(dm, "dm", (N, plan.D_out, plan.C)), _ptr(dx, "dx", (N, plan.D_in, plan.C)),
                                     _ptr(dvec, "dvec", (E, 3)), _ptr(ds, "ds", (E, plan.P, plan.C)),
                                     _stream(stream)), "e3_conv_bwd_noalloc")
    return dx, dvec, ds


def _optr(t, name, shape):
    return None if t is None else _ptr(t, name, shape)


@_on_stream
def conv_fwd_y(plan: Plan, graph: Graph, x, y, s, out=None, accumulate=False, stream=None):
    """m = conv(x, y, s) with the harmonics y [E, D_sh] given (m += ... when accumulate)."""
    N, E = graph.n_nodes, graph.n_edges
    out = _empty((N, plan.D_out, plan.C)) if out is None else out
    _check(lib().e3_conv_fwd_y(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C)),
                               _ptr(y, "y", (E, plan.D_sh)), _ptr(s, "s", (E, plan.P, plan.C)),
                               _ptr(out, "m", (N, plan.D_out, plan.C)), 1 if accumulate else 0, _stream(stream)),
           "e3_conv_fwd_y")
    return out


@_on_stream
def conv_bwd_y(plan: Plan, graph: Graph, x, y, s, dm, dx=None, dy=None, ds=None, want=("dx", "dy", "ds"),
               accumulate=False, ws=None, stream=None):
    """(dx, dy, ds) of eq. (conv-bwd) with y given; cotangents not in `want` are neither
    computed into memory nor returned (None)."""
    N, E = graph.n_nodes, graph.n_edges
    if "dx" in want and dx is None:
        dx = _empty((N, plan.D_in, plan.C))
    if "dy" in want and dy is None:
        dy = _empty((E, plan.D_sh))
    if "ds" in want and ds is None:
        ds = _empty((E, plan.P, plan.C))
    if ws is None:
        ws = workspace(conv_workspace_size(plan, graph)[1])
    _check(lib().e3_conv_bwd_y(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C)),
                               _ptr(y, "y", (E, plan.D_sh)), _ptr(s, "s", (E, plan.P, plan.C)),
                               _ptr(dm, "dm", (N, plan.D_out, plan.C)), _optr(dx, "dx", (N, plan.D_in, plan.C)),
                               _optr(dy, "dy", (E, plan.D_sh)), _optr(ds, "ds", (E, plan.P, plan.C)),
                               1 if accumulate else 0, ct.c_void_p(ws.data_ptr()), ws.numel(), _stream(stream)),
           "e3_conv_bwd_y")
    return dx, dy, ds


@_on_stream
def conv_bwd2(plan: Plan, graph: Graph, x, y, s, dm, ddx, ddy, dds, ws=None, stream=None):
    """Double backward: (gx, gy, gs, gdm), the variations of (x, y, s, dm) for
    variations (ddx, ddy, dds) of the backward's outputs."""
    N, E = graph.n_nodes, graph.n_edges
    gx, gdm = _empty((N, plan.D_in, plan.C)), _empty((N, plan.D_out, plan.C))
    gy, gs = _empty((E, plan.D_sh)), _empty((E, plan.P, plan.C))
    if ws is None:
        ws = workspace(conv_workspace_size(plan, graph)[1])
    _check(lib().e3_conv_bwd2(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C)),
                              _ptr(y, "y", (E, plan.D_sh)), _ptr(s, "s", (E, plan.P, plan.C)),
                              _ptr(dm, "dm", (N, plan.D_out, plan.C)), _ptr(ddx, "ddx", (N, plan.D_in, plan.C)),
                              _ptr(ddy, "ddy", (E, plan.D_sh)), _ptr(dds, "dds", (E, plan.P, plan.C)),
                              _ptr(gx, "gx", (N, plan.D_in, plan.C)), _ptr(gy, "gy", (E, plan.D_sh)),
                              _ptr(gs, "gs", (E, plan.P, plan.C)), _ptr(gdm, "gdm", (N, plan.D_out, plan.C)),
                              ct.c_void_p(ws.data_ptr()), ws.numel(), _stream(stream)), "e3_conv_bwd2")
    return gx, gy, gs, gdm


class RecordTP:
    """Tensor product with caller-supplied records (i0, i1, i2, value)."""

    def __init__(self, d_x: int, d_y: int, d_z: int, i0, i1, i2, val, y_per_channel: bool):
        i0, i1, i2 = (np.ascontiguousarray(a, dtype=np.int32) for a in (i0, i1, i2))
        val = np.ascontiguousarray(val, dtype=np.float64)
        h = ct.c_void_p()
        _check(lib().e3_tpg_create(d_x, d_y, d_z, val.shape[0], i0.ctypes.data_as(ct.c_void_p),
                                   i1.ctypes.data_as(ct.c_void_p), i2.ctypes.data_as(ct.c_void_p),
                                   val.ctypes.data_as(ct.c_void_p), 1 if y_per_channel else 0, ct.byref(h)),
               "e3_tpg_create")
        self.handle = h
        self.d_x, self.d_y, self.d_z, self.ypc = d_x, d_y, d_z, bool(y_per_channel)

    def close(self):
        if getattr(self, "handle", None) and self.handle.value:
            lib().e3_tpg_destroy(self.handle)
            self.handle = ct.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _yshape(self, R, C):
        return (R, self.d_y, C) if self.ypc else (R, self.d_y)

    @staticmethod
    def _kind(x):
        torch = _torch()
        return ("float64", "_f64") if x.dtype == torch.float64 else ("float32", "")

    @_on_stream
    def forward(self, x, y, out=None, stream=None):
        """z in the precision of x (float32 or float64)."""
        R, _, C = x.shape
        dt, sfx = self._kind(x)
        out = _torch().empty((R, self.d_z, C), dtype=x.dtype, device="cuda") if out is None else out
        _check(getattr(lib(), "e3_tpg_fwd" + sfx)(
            self.handle, _ptr(x, "x", (R, self.d_x, C), dt), _ptr(y, "y", self._yshape(R, C), dt),
            _ptr(out, "z", (R, self.d_z, C), dt), R, C, _stream(stream)), "e3_tpg_fwd" + sfx)
        return out

    @_on_stream
    def backward(self, x, y, dz, stream=None):
        R, _, C = x.shape
        dt, sfx = self._kind(x)
        torch = _torch()
        dx = torch.empty((R, self.d_x, C), dtype=x.dtype, device="cuda")
        dy = torch.empty(self._yshape(R, C), dtype=x.dtype, device="cuda")
        b = ct.c_size_t()
        _check(lib().e3_tpg_workspace_size(self.handle, R, C, ct.byref(b)), "e3_tpg_workspace_size")
        ws = workspace(b.value)
        _check(getattr(lib(), "e3_tpg_bwd" + sfx)(
            self.handle, _ptr(x, "x", (R, self.d_x, C), dt), _ptr(y, "y", self._yshape(R, C), dt),
            _ptr(dz, "dz", (R, self.d_z, C), dt), _ptr(dx, "dx", (R, self.d_x, C), dt),
            _ptr(dy, "dy", self._yshape(R, C), dt), ct.c_void_p(ws.data_ptr()), ws.numel(), R, C,
            _stream(stream)), "e3_tpg_bwd" + sfx)
        return dx, dy


class Linear:
    """Equivariant linear mixing between two irreps layouts (weights shared over m)."""

    def __init__(self, irreps_in: str, irreps_out: str):
        h = ct.c_void_p()
        _check(lib().e3_linear_create(irreps_in.encode(), irreps_out.encode(), ct.byref(h)), "e3_linear_create")
        self.handle = h
        nw, di, do, ci, co = ct.c_int64(), ct.c_int(), ct.c_int(), ct.c_int(), ct.c_int()
        _check(lib().e3_linear_query(h, ct.byref(nw), ct.byref(di), ct.byref(do), ct.byref(ci), ct.byref(co)),
               "e3_linear_query")
        self.n_weights, self.D_in, self.D_out, self.C_in, self.C_out = nw.value, di.value, do.value, ci.value, co.value

    def close(self):
        if getattr(self, "handle", None) and self.handle.value:
            lib().e3_linear_destroy(self.handle)
            self.handle = ct.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @_on_stream
    def forward(self, x, W, out=None, stream=None):
        n = x.shape[0]
        out = _empty((n, self.D_out, self.C_out)) if out is None else out
        _check(lib().e3_linear_fwd(self.handle, _ptr(x, "x", (n, self.D_in, self.C_in)),
                                   _ptr(W, "W", (self.n_weights,)), _ptr(out, "out", (n, self.D_out, self.C_out)),
                                   n, _stream(stream)), "e3_linear_fwd")
        return out

    def workspace_size(self) -> int:
        b = ct.c_size_t()
        _check(lib().e3_linear_workspace_size(self.handle, ct.byref(b)), "e3_linear_workspace_size")
        return b.value

    @_on_stream
    def backward(self, x, W, dout, dx=None, dW=None, ws=None, stream=None):
        n = x.shape[0]
        dx = _empty((n, self.D_in, self.C_in)) if dx is None else dx
        dW = _empty((self.n_weights,)) if dW is None else dW
        if ws is None:
            ws = workspace(self.workspace_size())
        _check(lib().e3_linear_bwd(self.handle, _ptr(x, "x", (n, self.D_in, self.C_in)),
                                   _ptr(W, "W", (self.n_weights,)), _ptr(dout, "dout", (n, self.D_out, self.C_out)),
                                   _ptr(dx, "dx", (n, self.D_in, self.C_in)), _ptr(dW, "dW", (self.n_weights,)),
                                   ct.c_void_p(ws.data_ptr()), ws.numel(), n, _stream(stream)), "e3_linear_bwd")
        return dx, dW


def conv_radial_workspace_size(plan: Plan, graph: Graph, K: int) -> int:
    b = ct.c_size_t()
    _check(lib().e3_conv_radial_workspace_size(plan.handle, graph.handle, K, ct.byref(b)),
           "e3_conv_radial_workspace_size")
    return b.value


@_on_stream
def conv_fwd_radial(plan: Plan, graph: Graph, x, vec, h, W, out=None, stream=None):
    """m with per-edge weights s_e = h_e W formed inside the kernel (h [E, K], W [K, P, C])."""
    N, E = graph.n_nodes, graph.n_edges
    K = W.shape[0]
    out = _empty((N, plan.D_out, plan.C)) if out is None else out
    _check(lib().e3_conv_fwd_radial(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C)),
                                    _ptr(vec, "vec", (E, 3)), _ptr(h, "h", (E, K)),
                                    _ptr(W, "W", (K, plan.P, plan.C)), K,
                                    _ptr(out, "m", (N, plan.D_out, plan.C)), _stream(stream)),
           "e3_conv_fwd_radial")
    return out


@_on_stream
def conv_bwd_radial(plan: Plan, graph: Graph, x, vec, h, W, dm, dx=None, dvec=None, dh=None, dW=None, ws=None,
                    stream=None):
    """(dx, dvec, dh, dW) of the convolution with fused radial weights."""
    N, E = graph.n_nodes, graph.n_edges
    K = W.shape[0]
    dx = _empty((N, plan.D_in, plan.C)) if dx is None else dx
    dvec = _empty((E, 3)) if dvec is None else dvec
    dh = _empty((E, K)) if dh is None else dh
    dW = _empty((K, plan.P, plan.C)) if dW is None else dW
    if ws is None:
        ws = workspace(conv_radial_workspace_size(plan, graph, K))
    _check(lib().e3_conv_bwd_radial(plan.handle, graph.handle, _ptr(x, "x", (N, plan.D_in, plan.C)),
                                    _ptr(vec, "vec", (E, 3)), _ptr(h, "h", (E, K)),
                                    _ptr(W, "W", (K, plan.P, plan.C)), K,
                                    _ptr(dm, "dm", (N, plan.D_out, plan.C)), _ptr(dx, "dx", (N, plan.D_in, plan.C)),
                                    _ptr(dvec, "dvec", (E, 3)), _ptr(dh, "dh", (E, K)),
                                    _ptr(dW, "dW", (K, plan.P, plan.C)), ct.c_void_p(ws.data_ptr()), ws.numel(),
                                    _stream(stream)), "e3_conv_bwd_radial")
    return dx, dvec, dh, dW


# ---------------------------------------------------------------- instrumentation
PROBE_NT_LOAD, PROBE_NT_STORE = 1, 2


@_on_stream
def probe_stream(src, dst, read_units: int, write_units: int, width: int, flags: int, stream=None):
    """One streaming probe launch; returns (bytes read, bytes written)."""
    br, bw = ct.c_size_t(), ct.c_size_t()
    sp = ct.c_void_p(src.data_ptr()) if src is not None else None
    dp = ct.c_void_p(dst.data_ptr()) if dst is not None else None
    sb = src.numel() * src.element_size() if src is not None else 0
    db = dst.numel() * dst.element_size() if dst is not None else 0
    _check(lib().e3_probe_stream(sp, sb, dp, db, read_units, write_units, width, flags, ct.byref(br),
                                 ct.byref(bw), _stream(stream)), "e3_probe_stream")
    return br.value, bw.value


# ---------------------------------------------------------------- timing
def timing_enable(on: bool = True):
    _check(lib().e3_timing_enable(1 if on else 0), "e3_timing_enable")


def timing_reset():
    _check(lib().e3_timing_reset(), "e3_timing_reset")


def timing_read() -> dict:
    """{kernel name: (summed ms, launches)} since the last reset."""
    n = ct.c_int()
    _check(lib().e3_timing_read(0, None, None, None, ct.byref(n)), "e3_timing_read")
    cap = n.value
    names = ct.create_string_buffer(32 * max(cap, 1))
    ms = np.zeros(max(cap, 1), np.float64)
    cnt = np.zeros(max(cap, 1), np.int64)
    _check(lib().e3_timing_read(cap, ct.cast(names, ct.c_void_p), ms.ctypes.data_as(ct.c_void_p),
                                cnt.ctypes.data_as(ct.c_void_p), ct.byref(n)), "e3_timing_read")
    out = {}
    for i in range(min(cap, n.value)):
        nm = names.raw[32 * i:32 * (i + 1)].split(b"\0", 1)[0].decode()
        out[nm] = (float(ms[i]), int(cnt[i]))
    return out
