"""Host-side harness of the CPU emulation library (test infrastructure).

Calls the same C ABI as paper_2607_18074_amd.api, with every device buffer in guarded host memory
(Dev): the emulated runtime places each buffer against inaccessible guard zones, so any access a
kernel makes outside it faults at once and is reported with the buffer, the offset, the kernel, the
block and the thread.  Never used by the package.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

from paper_2607_18074_amd import _lib
from tests.emu import build as _build

_L = None


def lib(asan=False):
    """The loaded emulation library (built on first use)."""
    global _L
    if _L is None:
        path = _build.build(asan=asan)
        L = ctypes.CDLL(path)
        for name, (res, args) in _lib._SIGNATURES.items():
            f = getattr(L, name, None)
            if f is not None:
                f.restype = res
                f.argtypes = args
        L.emu_galloc.restype = ctypes.c_void_p
        L.emu_galloc.argtypes = [ctypes.c_size_t, ctypes.c_char_p]
        L.emu_gfree.argtypes = [ctypes.c_void_p]
        L.emu_launch_count.restype = ctypes.c_long
        _L = L
    return _L


def check(rc):
    if rc != 0:
        raise _lib.SobekError(rc, lib().sobek_last_error().decode(errors="replace"))


class Dev:
    """A guarded 'device' buffer with a numpy view of its contents (filled with 0xff when created)."""

    def __init__(self, shape, dtype=np.float32, tag="buf", init=None):
        shape = tuple(int(s) for s in (shape if isinstance(shape, (tuple, list)) else (shape,)))
        self.shape, self.dtype = shape, np.dtype(dtype)
        n = int(np.prod(shape)) if shape else 1
        self.nbytes = n * self.dtype.itemsize
        self.ptr = lib().emu_galloc(self.nbytes, tag.encode())
        buf = (ctypes.c_char * max(self.nbytes, 1)).from_address(self.ptr)
        self.a = np.frombuffer(buf, dtype=self.dtype, count=n).reshape(shape)
        if init is not None:
            self.a[...] = init

    def np(self):
        return self.a.copy()

    # the few tensor methods the GPU test files call on their results
    def numel(self):
        return int(np.prod(self.shape)) if self.shape else 1

    def data_ptr(self):
        return self.ptr

    def cpu(self):
        return self

    def detach(self):
        return self

    def numpy(self):
        return self.a.copy()

    def fill_(self, v):
        self.a[...] = v
        return self

    def __rmul__(self, k):
        return Dev(self.shape, self.dtype, "scaled", k * self.a)


def dev(a, tag="in"):
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    return Dev(a.shape, a.dtype, tag, a)


def _p(d):
    # an empty tensor's data pointer is NULL
    return None if d is None or d.nbytes == 0 else ctypes.c_void_p(d.ptr)


class Plan:
    def __init__(self, irreps_in, lmax, irreps_out, K, layout="ir_mul", normalization="none", mode="uvw",
                 dtype="f32", policy="auto"):
        args = _lib._sig_args(irreps_in, lmax, irreps_out, K, layout, normalization, mode, dtype)
        h = ctypes.c_void_p()
        check(lib().sobek_plan_create(*args, ctypes.byref(h)))
        self.handle = h
        self.K = int(K)
        self.irreps_in = _lib.parse_irreps(irreps_in)
        self.irreps_out = _lib.parse_irreps(irreps_out)
        vals = [ctypes.c_int64() for _ in range(5)]
        check(lib().sobek_plan_info(h, *[ctypes.byref(v) for v in vals]))
        self.n_paths, self.n_weights, self.dim_in, self.dim_out, self.dim_sh = (v.value for v in vals)
        self.set_policy(policy)

    def set_policy(self, policy):
        check(lib().sobek_plan_set_policy(self.handle, {"all": 0, "groups": 1, "auto": 2}[policy]))
        self.policy = policy

    def paths(self):
        n = self.n_paths
        a, b, c = ((ctypes.c_int32 * n)() for _ in range(3))
        w = (ctypes.c_int64 * n)()
        check(lib().sobek_plan_paths(self.handle, a, b, c, w))
        return [(a[t], b[t], c[t], w[t]) for t in range(n)]

    def cg(self, path):
        i_in, i_sh, i_out, _ = self.paths()[path]
        li, ls, lo = self.irreps_in[i_in][1], i_sh, self.irreps_out[i_out][1]
        buf = (ctypes.c_double * ((2 * li + 1) * (2 * ls + 1) * (2 * lo + 1)))()
        check(lib().sobek_plan_cg(self.handle, path, buf))
        return np.array(buf).reshape(2 * li + 1, 2 * ls + 1, 2 * lo + 1)


class Graph:
    def __init__(self, rowptr, sender):
        rowptr = rowptr.a if isinstance(rowptr, Dev) else rowptr
        sender = sender.a if isinstance(sender, Dev) else sender
        self.rowptr = dev(np.asarray(rowptr, np.int32), "rowptr")
        self.sender = dev(np.asarray(sender, np.int32), "sender")
        self.N, self.E = len(rowptr) - 1, len(sender)
        nb = ctypes.c_size_t()
        check(lib().sobek_graph_prepare_size(self.N, self.E, ctypes.byref(nb)))
        self.buf = Dev(max(nb.value, 16), np.uint8, "graph buffer")
        h = ctypes.c_void_p()
        check(lib().sobek_graph_prepare(_p(self.rowptr), _p(self.sender), self.N, self.E, _p(self.buf), nb.value,
                                        ctypes.byref(h), None))
        self.handle = h
        self._ws = {}

    def workspace_bytes(self, plan, pass_, budget=0):
        nb = ctypes.c_size_t()
        check(lib().sobek_workspace_size(plan.handle, self.handle, _lib.PASSES[pass_], budget, ctypes.byref(nb)))
        return int(nb.value)

    def workspace(self, plan, pass_, budget=0):
        key = (id(plan), pass_, budget)
        if key not in self._ws:
            self._ws[key] = Dev(max(self.workspace_bytes(plan, pass_, budget), 256), np.uint8, f"workspace {pass_}")
        return self._ws[key]


def state_floats(plan, graph):
    nb = ctypes.c_size_t()
    check(lib().sobek_state_size(plan.handle, graph.handle, ctypes.byref(nb)))
    return int(nb.value) // 4


def new_state(plan, graph, device=None):
    return Dev(max(state_floats(plan, graph), 4), np.float32, "state")


def _ws(plan, graph, p, ws, budget):
    return graph.workspace(plan, p, budget) if ws is None else ws


def retention(plan, graph, budget=0):
    m, nb = ctypes.c_uint64(), ctypes.c_size_t()
    check(lib().sobek_retention_select(plan.handle, graph.handle, budget, ctypes.byref(m), ctypes.byref(nb)))
    return int(m.value), int(nb.value)


def kept_bytes(plan, graph, mask):
    nb = ctypes.c_size_t()
    check(lib().sobek_kept_size(plan.handle, graph.handle, mask, ctypes.byref(nb)))
    return int(nb.value)


def new_kept(plan, graph, mask, device=None):
    return Dev(max((kept_bytes(plan, graph, mask) + 3) // 4, 4), np.float32, "kept")


def conv_fwd(plan, graph, x, evec, phi, W, out=None, ws=None, budget=0, state=None, keep=None):
    out = Dev((graph.N, plan.dim_out), np.float32, "out") if out is None else out
    ws = _ws(plan, graph, "fwd", ws, budget)
    L = lib()
    if keep is not None:
        check(L.sobek_conv_fwd_keep(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(out), keep[0],
                                    _p(keep[1]), _p(ws), ws.nbytes, None))
    elif state is None:
        check(L.sobek_conv_fwd(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(out), _p(ws),
                               ws.nbytes, None))
    else:
        check(L.sobek_conv_fwd_save(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(out), _p(state),
                                    _p(ws), ws.nbytes, None))
    return out


def conv_bwd(plan, graph, x, evec, phi, W, gout, need=(True, True, True, True), ws=None, budget=0, state=None,
             adj_state=None, kept=None):
    N, E = graph.N, graph.E
    shapes = [(N, plan.dim_in), (E, 3), (E, plan.K), (plan.K, plan.n_weights)]
    outs = [Dev(s, np.float32, nm) if n else None for s, n, nm in zip(shapes, need, ("gx", "gevec", "gphi", "gW"))]
    ws = _ws(plan, graph, "bwd", ws, budget)
    L = lib()
    if kept is not None:
        check(L.sobek_conv_bwd_kept(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(gout), kept[0],
                                    _p(kept[1]), *[_p(o) for o in outs], _p(ws), ws.nbytes, None))
    elif state is None and adj_state is None:
        check(L.sobek_conv_bwd(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(gout),
                               *[_p(o) for o in outs], _p(ws), ws.nbytes, None))
    else:
        check(L.sobek_conv_bwd_saved(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(gout),
                                     _p(state), _p(adj_state), *[_p(o) for o in outs], _p(ws), ws.nbytes, None))
    return tuple(outs)


def conv_dbwd(plan, graph, x, evec, phi, W, gout, t_gx=None, t_gevec=None, t_gphi=None, t_gW=None,
              need=(True, True, True, True, True), ws=None, budget=0, adj_state=None):
    N, E = graph.N, graph.E
    shapes = [(N, plan.dim_out), (N, plan.dim_in), (E, 3), (E, plan.K), (plan.K, plan.n_weights)]
    names = ("g_gout", "g_x", "g_evec", "g_phi", "g_W")
    outs = [Dev(s, np.float32, nm) if n else None for s, n, nm in zip(shapes, need, names)]
    ws = _ws(plan, graph, "dbwd", ws, budget)
    L = lib()
    if adj_state is None:
        check(L.sobek_conv_dbwd(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(gout), _p(t_gx),
                                _p(t_gevec), _p(t_gphi), _p(t_gW), *[_p(o) for o in outs], _p(ws), ws.nbytes, None))
    else:
        check(L.sobek_conv_dbwd_saved(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(gout),
                                      _p(adj_state), _p(t_gx), _p(t_gevec), _p(t_gphi), _p(t_gW),
                                      *[_p(o) for o in outs], _p(ws), ws.nbytes, None))
    return tuple(outs)


def materialized_bytes(plan, graph, budget=0):
    nb = ctypes.c_size_t()
    check(lib().sobek_materialized_workspace_size(plan.handle, graph.handle, budget, ctypes.byref(nb)))
    return int(nb.value)


def conv_fwd_materialized(plan, graph, x, evec, phi, W, out=None, ws=None, budget=0):
    out = Dev((graph.N, plan.dim_out), np.float32, "out") if out is None else out
    if ws is None:
        ws = Dev(max(materialized_bytes(plan, graph, budget), 256), np.uint8, "materialized workspace")
    check(lib().sobek_conv_fwd_materialized(plan.handle, graph.handle, _p(x), _p(evec), _p(phi), _p(W), _p(out),
                                            _p(ws), ws.nbytes, None))
    return out


def launches():
    """Kernel launches the emulated runtime has run so far."""
    return int(lib().emu_launch_count())
