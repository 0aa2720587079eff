"""Torch-facing binding of libsobek_hip: plans, graphs, workspaces, autograd.

PyTorch supplies device memory and the current stream only; every step of the
operator runs in the library's HIP kernels.  Tensors must be contiguous fp32
(int32 for the CSR) CUDA tensors on the current device.
"""

from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import _lib
from ._lib import check, lib

_P = ctypes.c_void_p


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check_tensor(t, name, shape, dtype=torch.float32):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


POLICIES = {"all": 0, "groups": 1, "auto": 2}


class Plan:
    """Operator signature: irreps, spherical-harmonic order, radial width, channel mode ("uvw" fully
    connected, "uvu" channelwise), dtype ("f32", or "bf16_gemm": the channel GEMMs m = S A, A_bar =
    S^T mbar and, for multiplicities in multiples of 32 up to 128, Sbar = mbar A^T on bf16 MFMA with fp32
    accumulation; tensors stay fp32), and
    scratch policy ("all": every output group per receiver chunk; "groups": the receiver-state legs one
    output group at a time in chunks of n_g receivers, eq. receiver_chunk_budget; "auto", the default:
    "groups" for a pass whose all-group plan needs three or more receiver chunks, each too small to fill
    the GPU)."""

    def __init__(self, irreps_in, lmax, irreps_out, K, layout="ir_mul", normalization="none", mode="uvw",
                 dtype="f32", policy="auto"):
        self.irreps_in = _lib.parse_irreps(irreps_in)
        self.irreps_out = _lib.parse_irreps(irreps_out)
        self.lmax, self.K, self.layout, self.normalization = int(lmax), int(K), layout, normalization
        self.mode, self.dtype = mode, dtype
        args = _lib._sig_args(irreps_in, lmax, irreps_out, K, layout, normalization, mode, dtype)
        h = _P()
        check(lib().sobek_plan_create(*args, ctypes.byref(h)))
        self._h = h
        vals = [ctypes.c_int64() for _ in range(5)]
        check(lib().sobek_plan_info(h, *[ctypes.byref(v) for v in vals]))
        self.n_paths, self.n_weights, self.dim_in, self.dim_out, self.dim_sh = (v.value for v in vals)
        self.policy = "auto"
        self.set_policy(policy)

    def set_policy(self, policy):
        check(lib().sobek_plan_set_policy(self._h, POLICIES[policy]))
        self.policy = policy

    @property
    def handle(self):
        return self._h

    def paths(self):
        n = self.n_paths
        a, b, c = ((ctypes.c_int32 * n)() for _ in range(3))
        w = (ctypes.c_int64 * n)()
        check(lib().sobek_plan_paths(self._h, a, b, c, w))
        return [(a[t], b[t], c[t], w[t]) for t in range(n)]

    def cg(self, path):
        i_in, i_sh, i_out, _ = self.paths()[path]
        li, ls, lo = self.irreps_in[i_in][1], i_sh, self.irreps_out[i_out][1]
        buf = (ctypes.c_double * ((2 * li + 1) * (2 * ls + 1) * (2 * lo + 1)))()
        check(lib().sobek_plan_cg(self._h, path, buf))
        return np.array(buf).reshape(2 * li + 1, 2 * ls + 1, 2 * lo + 1)

    def weight_std(self):
        """Per-column std 1/sqrt(K * fan_in) of the weight init (fan_in = terms summed into one output
        channel: the sum of C_in over the paths into the output irrep for uvw, their number for uvu)."""
        fan = {}
        paths = self.paths()
        uvu = self.mode == "uvu"
        for (a, _b, c, _w) in paths:
            fan[c] = fan.get(c, 0) + (1 if uvu else self.irreps_in[a][0])
        std = np.zeros(self.n_weights)
        for (a, _b, c, w) in paths:
            n = self.irreps_in[a][0] * (1 if uvu else self.irreps_out[c][0])
            std[w:w + n] = 1.0 / np.sqrt(self.K * fan[c])
        return std

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            try:
                lib().sobek_plan_destroy(h)
            except Exception:
                pass
            self._h = None


class Graph:
    """Receiver-sorted CSR on the device plus its prepared sender-sorted view."""

    def __init__(self, rowptr, sender):
        if rowptr.dtype != torch.int32 or sender.dtype != torch.int32:
            raise ValueError("rowptr and sender must be int32")
        self.rowptr, self.sender = rowptr.contiguous(), sender.contiguous()
        self.N, self.E = int(rowptr.shape[0]) - 1, int(sender.shape[0])
        nb = ctypes.c_size_t()
        check(lib().sobek_graph_prepare_size(self.N, self.E, ctypes.byref(nb)))
        self.buf = torch.empty(max(int(nb.value), 16), dtype=torch.uint8, device=rowptr.device)
        h = _P()
        check(lib().sobek_graph_prepare(_ptr(self.rowptr), _ptr(self.sender), self.N, self.E, _ptr(self.buf),
                                        nb.value, ctypes.byref(h), _stream()))
        self._h = h
        self._ws = {}

    @property
    def handle(self):
        return self._h

    def workspace_bytes(self, plan, pass_, budget=0):
        """sobek_workspace_size of a pass ("fwd", "bwd", "dbwd") at `budget` bytes (0 = the default; 1 gives
        the minimum, chunks of one receiver)."""
        nb = ctypes.c_size_t()
        check(lib().sobek_workspace_size(plan.handle, self._h, _lib.PASSES[pass_], budget, ctypes.byref(nb)))
        return int(nb.value)

    def workspace(self, plan, pass_, budget=0):
        """Cached workspace tensor for (plan, pass, budget)."""
        key = (id(plan), pass_, budget)
        if key not in self._ws:
            nb = self.workspace_bytes(plan, pass_, budget)
            self._ws[key] = torch.empty(max(nb, 256), dtype=torch.uint8, device=self.rowptr.device)
        return self._ws[key]

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            try:
                lib().sobek_graph_destroy(h)
            except Exception:
                pass
            self._h = None


def _ws(plan, graph, pass_, ws, budget):
    if ws is None:
        ws = graph.workspace(plan, pass_, budget)
    return ws


def state_floats(plan, graph):
    """Length of the retained receiver state of `graph` (fp32 elements; node-bounded)."""
    nb = ctypes.c_size_t()
    check(lib().sobek_state_size(plan.handle, graph.handle, ctypes.byref(nb)))
    return int(nb.value) // 4


def new_state(plan, graph, device=None):
    """An uninitialised buffer for the retained receiver state."""
    return torch.empty(max(state_floats(plan, graph), 4), dtype=torch.float32,
                       device=device or graph.rowptr.device)


def _check_state(plan, graph, state):
    if state is not None:
        _check_tensor(state, "state", (state.numel(),))
        if state.numel() < state_floats(plan, graph):
            raise ValueError("state buffer is smaller than sobek_state_size")


def retention(plan, graph, budget=0):
    """(group mask, kept bytes) of the output groups whose state the forward keeps within `budget` bytes
    (0 = 1 GiB): the subset that avoids the most recomputed coupling work, ties to fewer bytes."""
    m, nb = ctypes.c_uint64(), ctypes.c_size_t()
    check(lib().sobek_retention_select(plan.handle, graph.handle, budget, ctypes.byref(m), ctypes.byref(nb)))
    return int(m.value), int(nb.value)


def kept_bytes(plan, graph, mask):
    nb = ctypes.c_size_t()
    check(lib().sobek_kept_size(plan.handle, graph.handle, mask, ctypes.byref(nb)))
    return int(nb.value)


def new_kept(plan, graph, mask, device=None):
    """An uninitialised buffer for the kept state of the output groups in `mask` (as 4-byte words)."""
    return torch.empty(max((kept_bytes(plan, graph, mask) + 3) // 4, 4), dtype=torch.float32,
                       device=device or graph.rowptr.device)


def _check_kept(plan, graph, kept):
    if kept is not None:
        mask, buf = kept
        _check_tensor(buf, "kept", (buf.numel(),))
        if buf.numel() * 4 < kept_bytes(plan, graph, mask):
            raise ValueError("kept buffer is smaller than sobek_kept_size")


def conv_fwd(plan, graph, x, evec, phi, W, out=None, ws=None, budget=0, state=None, keep=None):
    """m = conv(x, evec, phi, W); with `state` (from new_state) S of every receiver is kept in it; with
    keep = (mask, buffer from new_kept) the state of the output groups in mask is kept there."""
    N, E = graph.N, graph.E
    _check_tensor(x, "x", (N, plan.dim_in))
    _check_tensor(evec, "evec", (E, 3))
    _check_tensor(phi, "phi", (E, plan.K))
    _check_tensor(W, "W", (plan.K, plan.n_weights))
    _check_state(plan, graph, state)
    if out is None:
        out = torch.empty(N, plan.dim_out, dtype=torch.float32, device=x.device)
    _check_tensor(out, "out", (N, plan.dim_out))
    ws = _ws(plan, graph, "fwd", ws, budget)
    _check_kept(plan, graph, keep)
    if keep is not None:
        check(lib().sobek_conv_fwd_keep(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W),
                                        _ptr(out), keep[0], _ptr(keep[1]), _ptr(ws), ws.numel(), _stream()))
    elif state is None:
        check(lib().sobek_conv_fwd(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W), _ptr(out),
                                   _ptr(ws), ws.numel(), _stream()))
    else:
        check(lib().sobek_conv_fwd_save(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W),
                                        _ptr(out), _ptr(state), _ptr(ws), ws.numel(), _stream()))
    return out


def materialized_bytes(plan, graph, budget=0):
    """Workspace bytes of the materialized forward: W and the edge messages for every edge (budget 0), or
    `budget` bytes of edge windows (at least one receiver's edges)."""
    nb = ctypes.c_size_t()
    check(lib().sobek_materialized_workspace_size(plan.handle, graph.handle, budget, ctypes.byref(nb)))
    return int(nb.value)


def conv_fwd_materialized(plan, graph, x, evec, phi, W, out=None, ws=None, budget=0):
    """The materialized forward (W = phi A and the edge messages formed in the workspace, then summed per
    receiver): the conventional evaluation order the streamed forward avoids, same result."""
    N, E = graph.N, graph.E
    _check_tensor(x, "x", (N, plan.dim_in))
    _check_tensor(evec, "evec", (E, 3))
    _check_tensor(phi, "phi", (E, plan.K))
    _check_tensor(W, "W", (plan.K, plan.n_weights))
    if out is None:
        out = torch.empty(N, plan.dim_out, dtype=torch.float32, device=x.device)
    _check_tensor(out, "out", (N, plan.dim_out))
    if ws is None:
        ws = torch.empty(max(materialized_bytes(plan, graph, budget), 256), dtype=torch.uint8, device=x.device)
    check(lib().sobek_conv_fwd_materialized(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W),
                                            _ptr(out), _ptr(ws), ws.numel(), _stream()))
    return out


def conv_bwd(plan, graph, x, evec, phi, W, gout, need=(True, True, True, True), ws=None, budget=0, state=None,
             adj_state=None, kept=None):
    """(gx, gevec, gphi, gW); entries not in `need` are None.

    `state`: the retained receiver state of conv_fwd(..., state=...) with the same x, evec and phi; the
    weight gradient then reads it instead of recomputing S.  `adj_state` (from new_state): receives the
    adjoint state Sbar = gout A^T of every receiver, for conv_dbwd(..., adj_state=...).  `kept`: the
    (mask, buffer) of conv_fwd(..., keep=...); the weight gradient reads those groups and recomputes the
    others one group at a time.
    """
    N, E = graph.N, graph.E
    _check_tensor(x, "x", (N, plan.dim_in))
    _check_tensor(evec, "evec", (E, 3))
    _check_tensor(phi, "phi", (E, plan.K))
    _check_tensor(W, "W", (plan.K, plan.n_weights))
    _check_tensor(gout, "gout", (N, plan.dim_out))
    dev = x.device
    shapes = [(N, plan.dim_in), (E, 3), (E, plan.K), (plan.K, plan.n_weights)]
    outs = [torch.empty(s, dtype=torch.float32, device=dev) if n else None for s, n in zip(shapes, need)]
    _check_state(plan, graph, state)
    _check_state(plan, graph, adj_state)
    ws = _ws(plan, graph, "bwd", ws, budget)
    _check_kept(plan, graph, kept)
    if kept is not None:
        if state is not None or adj_state is not None:
            raise ValueError("kept groups do not combine with state or adj_state")
        check(lib().sobek_conv_bwd_kept(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W),
                                        _ptr(gout), kept[0], _ptr(kept[1]), *[_ptr(o) for o in outs], _ptr(ws),
                                        ws.numel(), _stream()))
    elif state is None and adj_state is None:
        check(lib().sobek_conv_bwd(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W), _ptr(gout),
                                   *[_ptr(o) for o in outs], _ptr(ws), ws.numel(), _stream()))
    else:
        check(lib().sobek_conv_bwd_saved(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W),
                                         _ptr(gout), _ptr(state), _ptr(adj_state), *[_ptr(o) for o in outs],
                                         _ptr(ws), ws.numel(), _stream()))
    return tuple(outs)


def conv_dbwd(plan, graph, x, evec, phi, W, gout, t_gx=None, t_gevec=None, t_gphi=None, t_gW=None,
              need=(True, True, True, True, True), ws=None, budget=0, adj_state=None):
    """(g_gout, g_x, g_evec, g_phi, g_W); entries not in `need` are None.

    `adj_state`: the adjoint state kept by conv_bwd(..., adj_state=...) with the same gout and W.
    """
    N, E = graph.N, graph.E
    _check_tensor(x, "x", (N, plan.dim_in))
    _check_tensor(evec, "evec", (E, 3))
    _check_tensor(phi, "phi", (E, plan.K))
    _check_tensor(W, "W", (plan.K, plan.n_weights))
    _check_tensor(gout, "gout", (N, plan.dim_out))
    _check_tensor(t_gx, "t_gx", (N, plan.dim_in))
    _check_tensor(t_gevec, "t_gevec", (E, 3))
    _check_tensor(t_gphi, "t_gphi", (E, plan.K))
    _check_tensor(t_gW, "t_gW", (plan.K, plan.n_weights))
    dev = x.device
    shapes = [(N, plan.dim_out), (N, plan.dim_in), (E, 3), (E, plan.K), (plan.K, plan.n_weights)]
    outs = [torch.empty(s, dtype=torch.float32, device=dev) if n else None for s, n in zip(shapes, need)]
    _check_state(plan, graph, adj_state)
    ws = _ws(plan, graph, "dbwd", ws, budget)
    if adj_state is None:
        check(lib().sobek_conv_dbwd(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W), _ptr(gout),
                                    _ptr(t_gx), _ptr(t_gevec), _ptr(t_gphi), _ptr(t_gW), *[_ptr(o) for o in outs],
                                    _ptr(ws), ws.numel(), _stream()))
    else:
        check(lib().sobek_conv_dbwd_saved(plan.handle, graph.handle, _ptr(x), _ptr(evec), _ptr(phi), _ptr(W),
                                          _ptr(gout), _ptr(adj_state), _ptr(t_gx), _ptr(t_gevec), _ptr(t_gphi),
                                          _ptr(t_gW), *[_ptr(o) for o in outs], _ptr(ws), ws.numel(), _stream()))
    return tuple(outs)


# ---------------------------------------------------------------------------
# autograd: forward -> backward -> double backward (a third order raises)
# ---------------------------------------------------------------------------

def _c(t):
    return None if t is None else t.contiguous()


class _TPConvBackward(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, evec, phi, W, gout, plan, graph, state):
        ctx.plan, ctx.graph = plan, graph
        ctx.save_for_backward(x, evec, phi, W, gout)
        # with retention, the adjoint state is kept for the double backward as well
        ctx.adj_state = new_state(plan, graph, x.device) if state is not None else None
        return conv_bwd(plan, graph, x, evec, phi, W, gout, state=state, adj_state=ctx.adj_state)

    @staticmethod
    def backward(ctx, t_gx, t_gevec, t_gphi, t_gW):
        x, evec, phi, W, gout = ctx.saved_tensors
        g_gout, g_x, g_evec, g_phi, g_W = conv_dbwd(ctx.plan, ctx.graph, x, evec, phi, W, gout, _c(t_gx),
                                                    _c(t_gevec), _c(t_gphi), _c(t_gW), adj_state=ctx.adj_state)
        return g_x, g_evec, g_phi, g_W, g_gout, None, None, None


class TPConv(torch.autograd.Function):
    """m = conv(x, evec, phi, W) with first and second derivatives through the library."""

    @staticmethod
    def forward(ctx, x, evec, phi, W, plan, graph, retain_state):
        ctx.plan, ctx.graph = plan, graph
        ctx.save_for_backward(x, evec, phi, W)
        ctx.state = new_state(plan, graph, x.device) if retain_state else None
        return conv_fwd(plan, graph, x, evec, phi, W, state=ctx.state)

    @staticmethod
    def backward(ctx, gout):
        x, evec, phi, W = ctx.saved_tensors
        gx, gevec, gphi, gW = _TPConvBackward.apply(x, evec, phi, W, gout.contiguous(), ctx.plan, ctx.graph,
                                                    ctx.state)
        return gx, gevec, gphi, gW, None, None, None


def tp_conv(plan, graph, x, evec, phi, W, retain_state=False):
    """Differentiable convolution.  retain_state=True keeps S of every receiver from the forward, and Sbar of
    every receiver from the backward (each sobek_state_size bytes, node-bounded), so that neither the
    backward's weight gradient nor the double backward recomputes them."""
    return TPConv.apply(x, evec, phi, W, plan, graph, bool(retain_state))
