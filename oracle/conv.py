"""Forward, backward and double backward of the edge-conditioned TP convolution.

Test infrastructure only (see ``oracle/__init__``).  Float64 throughout; the
caller passes the same (fp32 or bf16-rounded) values the GPU receives, and they
are upcast here.

Materialised route (the plain definition)
-----------------------------------------
Forward, §2.4 eqs. ``standard_tpconv_background`` and
``radial_projection_background``: per edge chunk the weights W_e = phi_e A are
formed, every path's unweighted angular contraction

    C[e, u, m_o] = sum_{m_i, m_y} c^pi[m_i, m_y, m_o] x_{j(e)}[u, m_i] Y_e[m_y]

(§4.2 eq. ``angular_path_contraction``) is mixed into a per-edge message
msg[e, w, m_o] = sum_u W_e[pi, u, w] C[e, u, m_o], and messages are summed into
their receivers.

Backward, §3.2: h = <m_bar_i, T> (eq. ``streamed_weight_adjoint``), A_bar =
sum phi h and phi_bar = A h (eq. ``streamed_radial_adjoints``), x_bar and Y_bar
through the adjoints of the two partial Jacobians (eq.
``streamed_operand_adjoints``); edge-vector gradients follow by the chain rule
through the SH Jacobian, r_bar = J^T Y_bar.

Double backward, §3.3: the vector-Jacobian product of the backward map
(m_bar, x, evec, phi, A) -> (x_bar, evec_bar, phi_bar, A_bar) with cotangents
(x_dot, evec_dot, phi_dot, A_dot).  With Y_dot = J evec_dot, w_dot = phi_dot A +
phi A_dot and T_dot = T(x_dot, Y) + T(x, Y_dot) (eq.
``streamed_directional_terms``), the outputs are the paper's dotted quantities
with no direction on m_bar: the tangent output m_dot (eq.
``streamed_second_order_local_terms``) is the gradient for m_bar; the radial
and operand gradients are eqs. ``streamed_radial_second_adjoints`` and
``streamed_operand_second_adjoints``.  Because the operator here takes edge
vectors rather than Y, the edge-vector gradient has one extra chain term the
paper's Y-input operator does not have:
    g_evec = J^T g_Y + sum_m Y_bar_m Hess(Y_m) evec_dot.

Channel modes (§2.3): fully connected ``uvw`` (eq. ``uvw_connection``) mixes
every input channel u into every output channel w of a path with the C_in x
C_out block W_e[pi, u, w]; channelwise ``uvu`` (eq. ``uvu_connection``) ties
output channel u to input channel u with one weight W_e[pi, u] (C_out = C_in).
Only the per-path mixing (``_apply`` and its two transposes) depends on the mode.

Receiver route (cross-check of the reassociation)
-------------------------------------------------
§4.2-§4.4: S_i = sum_e phi_e (x) C_e (eq. ``receiver_state``), m = S A (eq.
``receiver_matrix_product``), S_bar = m_bar A^T and A_bar = S^T m_bar (eq.
``receiver_adjoint``), and the product rules of eq. ``receiver_double_adjoint``
with d m_bar = 0.  Exact arithmetic makes it equal to the materialised route.

Graph: receiver-sorted CSR (rowptr[N+1], sender[E]); edge arrays (evec, phi)
are in the same edge order; evec = r_sender - r_receiver (§2.4).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import cg as _cg
from . import irreps as _ir
from . import sh as _sh


@dataclass
class Problem:
    irreps_in: list
    lmax: int
    irreps_out: list
    K: int
    normalization: str = "none"
    layout: str = "ir_mul"
    mode: str = "uvw"           # "uvw": eq. uvw_connection; "uvu": eq. uvu_connection
    paths: list = field(init=False)
    coeffs: list = field(init=False)
    irreps_sh: list = field(init=False)
    n_w: int = field(init=False)

    def __post_init__(self):
        self.irreps_in = _ir.parse_irreps(self.irreps_in)
        self.irreps_out = _ir.parse_irreps(self.irreps_out)
        self.irreps_sh = _ir.sh_irreps(self.lmax)
        self.paths = _ir.enumerate_paths(self.irreps_in, self.irreps_sh, self.irreps_out, self.mode)
        self.coeffs = _cg.path_coefficients(self.paths, self.normalization, self.mode)
        self.n_w = _ir.num_weights(self.paths)

    @property
    def dim_in(self):
        return _ir.dim(self.irreps_in)

    @property
    def dim_out(self):
        return _ir.dim(self.irreps_out)


def receivers_from_rowptr(rowptr):
    rowptr = np.asarray(rowptr, dtype=np.int64)
    n = len(rowptr) - 1
    return np.repeat(np.arange(n, dtype=np.int64), np.diff(rowptr))


def _chunks(E, n_w, budget_bytes=256 << 20):
    step = max(1, int(budget_bytes // (8 * max(n_w, 1) * 3)))
    for s in range(0, E, step):
        yield s, min(E, s + step)


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def _sh_slice(Y, l):
    return Y[:, l * l:(l + 1) * (l + 1)]


def _contract_y(c, Yb):
    """M[e, m_i, m_o] = sum_{m_y} c[m_i, m_y, m_o] Y[e, m_y]."""
    return np.einsum("ijk,ej->eik", c, Yb)


def _prepare(prob, x, rowptr, sender):
    xb = _ir.flat_to_blocks(_f64(x), prob.irreps_in, prob.layout)
    recv = receivers_from_rowptr(rowptr)
    send = np.asarray(sender, dtype=np.int64)
    return xb, recv, send


# ---------------------------------------------------------------------------
# channel mixing of one path (§2.3): fully connected, eq. uvw_connection,
# z_w = sum_u W[u, w] T_u; channelwise, eq. uvu_connection, z_u = W[u] T_u
# ---------------------------------------------------------------------------

def _w_path(prob, We, p):
    """Per-edge weights of path p: [e, C_in, C_out] (uvw) or [e, C_in] (uvu)."""
    sl = We[:, p["w_off"]:p["w_off"] + p["n_w"]]
    return sl.reshape(len(We), p["c_in"], p["c_out"]) if prob.mode == "uvw" else sl


def _apply(prob, Wp, T):
    """Message [e, C_out, d_out] of path weights Wp on unweighted contractions T [e, C_in, d_out]."""
    return np.matmul(np.swapaxes(Wp, 1, 2), T) if prob.mode == "uvw" else Wp[:, :, None] * T


def _apply_T(prob, Wp, G):
    """Transpose of _apply in T: D [e, C_in, d_out] from a message-shaped G [e, C_out, d_out]."""
    return np.matmul(Wp, G) if prob.mode == "uvw" else Wp[:, :, None] * G


def _weight_adj(prob, T, G):
    """Transpose of _apply in the weights: h [e, n_w of the path] = d<G, _apply(W, T)>/dW."""
    if prob.mode == "uvw":
        return np.matmul(T, np.swapaxes(G, 1, 2)).reshape(len(T), -1)
    return np.einsum("eum,eum->eu", T, G)


# ---------------------------------------------------------------------------
# materialised route
# ---------------------------------------------------------------------------

def fwd(prob, x, evec, phi, W, rowptr, sender):
    """m[N, C_out] (flat, prob.layout)."""
    xb, recv, send = _prepare(prob, x, rowptr, sender)
    evec, phi, W = _f64(evec), _f64(phi), _f64(W)
    N = len(rowptr) - 1
    mb = [np.zeros((N, mul, 2 * l + 1)) for (mul, l, _p) in prob.irreps_out]
    for s, t in _chunks(len(send), prob.n_w):
        Y = _sh.sh(prob.lmax, evec[s:t])
        We = phi[s:t] @ W                                  # edge weights, eq. radial_projection_background
        for p, c in zip(prob.paths, prob.coeffs):
            Wp = _w_path(prob, We, p)
            xs = xb[p["i_in"]][send[s:t]]                    # [e, C_in, d_in]
            Ct = np.matmul(xs, _contract_y(c, _sh_slice(Y, p["l_sh"])))   # [e, C_in, d_out]
            msg = _apply(prob, Wp, Ct)                     # [e, C_out, d_out]
            np.add.at(mb[p["i_out"]], recv[s:t], msg)
    return _ir.blocks_to_flat(mb, prob.irreps_out, prob.layout)



def bwd(prob, x, evec, phi, W, rowptr, sender, gout):
    """dict(gx, gevec, gphi, gW): gradients of <gout, fwd(...)>."""
    xb, recv, send = _prepare(prob, x, rowptr, sender)
    evec, phi, W = _f64(evec), _f64(phi), _f64(W)
    gb = _ir.flat_to_blocks(_f64(gout), prob.irreps_out, prob.layout)
    N, E = len(rowptr) - 1, len(send)
    gxb = [np.zeros_like(b) for b in xb]
    gW = np.zeros_like(W)
    gphi = np.zeros((E, prob.K))
    gevec = np.zeros((E, 3))
    nsh = (prob.lmax + 1) ** 2
    for s, t in _chunks(E, prob.n_w):
        e = t - s
        Y = _sh.sh(prob.lmax, evec[s:t])
        J = _sh.sh_jacobian(prob.lmax, evec[s:t])
        We = phi[s:t] @ W
        h = np.zeros((e, prob.n_w))
        gY = np.zeros((e, nsh))
        for p, c in zip(prob.paths, prob.coeffs):
            Wp = _w_path(prob, We, p)
            Yb = _sh_slice(Y, p["l_sh"])
            M = _contract_y(c, Yb)
            xs = xb[p["i_in"]][send[s:t]]
            Ct = np.matmul(xs, M)                          # T(x_j, Y) unweighted
            gr = gb[p["i_out"]][recv[s:t]]                 # m_bar of the receiver [e, C_out, d_out]
            # h[e, u, w] = <m_bar_i, T_{pi,(u,w)}>      (eq. streamed_weight_adjoint)
            h[:, p["w_off"]:p["w_off"] + p["n_w"]] = _weight_adj(prob, Ct, gr)
            # D[e, u, m_o] = sum_w W_e[u, w] m_bar[w, m_o]
            D = _apply_T(prob, Wp, gr)
            # x_bar_j += D_x T^* : sum_{m_y, m_o} c Y D        (eq. streamed_operand_adjoints)
            np.add.at(gxb[p["i_in"]], send[s:t], np.matmul(D, np.swapaxes(M, 1, 2)))
            # Y_bar += D_Y T^* : sum_{m_i, m_o, u} c x D
            P = np.matmul(np.swapaxes(xs, 1, 2), D)        # [e, d_in, d_out]
            l = p["l_sh"]
            gY[:, l * l:(l + 1) ** 2] += np.einsum("ijk,eik->ej", c, P)
        gW += phi[s:t].T @ h                               # A_bar = sum phi h    (eq. streamed_radial_adjoints)
        gphi[s:t] = h @ W.T                                # phi_bar = A h
        gevec[s:t] = np.einsum("ej,ejk->ek", gY, J)        # chain rule through the SH
    return dict(gx=_ir.blocks_to_flat(gxb, prob.irreps_in, prob.layout), gevec=gevec, gphi=gphi, gW=gW)


def dbwd(prob, x, evec, phi, W, rowptr, sender, gout,
         t_gx=None, t_gevec=None, t_gphi=None, t_gW=None):
    """VJP of bwd with cotangents for (gx, gevec, gphi, gW); None means zero.

    Returns dict(g_gout, g_x, g_evec, g_phi, g_W).
    """
    xb, recv, send = _prepare(prob, x, rowptr, sender)
    evec, phi, W = _f64(evec), _f64(phi), _f64(W)
    gb = _ir.flat_to_blocks(_f64(gout), prob.irreps_out, prob.layout)
    N, E = len(rowptr) - 1, len(send)
    xdb = (_ir.flat_to_blocks(_f64(t_gx), prob.irreps_in, prob.layout)
           if t_gx is not None else [np.zeros_like(b) for b in xb])
    rdot = _f64(t_gevec) if t_gevec is not None else np.zeros((E, 3))
    phid = _f64(t_gphi) if t_gphi is not None else np.zeros((E, prob.K))
    Wd = _f64(t_gW) if t_gW is not None else np.zeros_like(W)

    out_m = [np.zeros((N, mul, 2 * l + 1)) for (mul, l, _p) in prob.irreps_out]
    g_xb = [np.zeros_like(b) for b in xb]
    g_W = np.zeros_like(W)
    g_phi = np.zeros((E, prob.K))
    g_evec = np.zeros((E, 3))
    nsh = (prob.lmax + 1) ** 2
    for s, t in _chunks(E, prob.n_w):
        e = t - s
        Y = _sh.sh(prob.lmax, evec[s:t])
        J = _sh.sh_jacobian(prob.lmax, evec[s:t])
        Hs = _sh.sh_hessian(prob.lmax, evec[s:t])
        Yd = np.einsum("ejk,ek->ej", J, rdot[s:t])                  # Y_dot = J evec_dot
        We = phi[s:t] @ W
        Wed = phid[s:t] @ W + phi[s:t] @ Wd                          # w_dot = phi_dot A + phi A_dot
        h = np.zeros((e, prob.n_w))
        hd = np.zeros((e, prob.n_w))
        gY = np.zeros((e, nsh))
        Ybar = np.zeros((e, nsh))
        for p, c in zip(prob.paths, prob.coeffs):
            sl = slice(p["w_off"], p["w_off"] + p["n_w"])
            Wp = _w_path(prob, We, p)
            Wdp = _w_path(prob, Wed, p)
            l = p["l_sh"]
            M = _contract_y(c, _sh_slice(Y, l))
            Md = _contract_y(c, _sh_slice(Yd, l))
            xs = xb[p["i_in"]][send[s:t]]
            xds = xdb[p["i_in"]][send[s:t]]
            Ct = np.matmul(xs, M)                                     # T(x, Y)
            Ctd = np.matmul(xds, M) + np.matmul(xs, Md)               # T_dot = T(x_dot, Y) + T(x, Y_dot)
            gr = gb[p["i_out"]][recv[s:t]]
            # tangent output m_dot = sum (w_dot T + w T_dot)  -> gradient for m_bar
            msg = _apply(prob, Wdp, Ct) + _apply(prob, Wp, Ctd)
            np.add.at(out_m[p["i_out"]], recv[s:t], msg)
            h[:, sl] = _weight_adj(prob, Ct, gr)
            hd[:, sl] = _weight_adj(prob, Ctd, gr)                    # h_dot = <m_bar, T_dot>
            D = _apply_T(prob, Wp, gr)
            Dd = _apply_T(prob, Wdp, gr)
            # x_bar_dot = sum (w_dot B^x + w B_dot^x), B_dot^x = D_x T(., Y_dot)^* m_bar
            np.add.at(g_xb[p["i_in"]], send[s:t],
                      np.matmul(Dd, np.swapaxes(M, 1, 2)) + np.matmul(D, np.swapaxes(Md, 1, 2)))
            # Y_bar_dot = sum (w_dot B^Y + w B_dot^Y), B_dot^Y = D_Y T(x_dot, .)^* m_bar
            Pd = np.matmul(np.swapaxes(xs, 1, 2), Dd) + np.matmul(np.swapaxes(xds, 1, 2), D)
            gY[:, l * l:(l + 1) ** 2] += np.einsum("ijk,eik->ej", c, Pd)
            P = np.matmul(np.swapaxes(xs, 1, 2), D)
            Ybar[:, l * l:(l + 1) ** 2] += np.einsum("ijk,eik->ej", c, P)
        g_W += phid[s:t].T @ h + phi[s:t].T @ hd                    # A_bar_dot
        g_phi[s:t] = h @ Wd.T + hd @ W.T                             # phi_bar_dot
        g_evec[s:t] = (np.einsum("ej,ejk->ek", gY, J)
                       + np.einsum("ej,ejkl,el->ek", Ybar, Hs, rdot[s:t]))
    return dict(g_gout=_ir.blocks_to_flat(out_m, prob.irreps_out, prob.layout),
                g_x=_ir.blocks_to_flat(g_xb, prob.irreps_in, prob.layout),
                g_evec=g_evec, g_phi=g_phi, g_W=g_W)


# ---------------------------------------------------------------------------
# receiver-factorised route (cross-check of the reassociation)
# ---------------------------------------------------------------------------

def _edge_C(prob, xb, Y, send):
    """C[pi] = [E, C_in, d_out] unweighted angular contractions."""
    out = []
    for p, c in zip(prob.paths, prob.coeffs):
        M = _contract_y(c, _sh_slice(Y, p["l_sh"]))
        out.append(np.matmul(xb[p["i_in"]][send], M))
    return out


def _receiver_state(prob, phi, Cs, recv, N):
    """S[pi] = [N, K, C_in, d_out] = sum_e phi_e (x) C_e   (eq. receiver_state)."""
    S = []
    for p, Ct in zip(prob.paths, Cs):
        Sp = np.zeros((N, prob.K, p["c_in"], 2 * p["l_out"] + 1))
        np.add.at(Sp, recv, phi[:, :, None, None] * Ct[:, None, :, :])
        S.append(Sp)
    return S


def _A(prob, W, p):
    """A_pi: [K, C_in, C_out] (uvw) or [K, C_in] (uvu) view of the flattened weights."""
    Wp = W[:, p["w_off"]:p["w_off"] + p["n_w"]]
    return Wp.reshape(prob.K, p["c_in"], p["c_out"]) if prob.mode == "uvw" else Wp


def _state_times_A(prob, Sp, A):
    """Receiver mixing of one path: m[n, w, m_o] = sum_{q, u} S[n, q, u, m_o] A[q, u, w] (uvw);
    m[n, u, m_o] = sum_q S[n, q, u, m_o] A[q, u] (uvu)."""
    return np.einsum("nqum,quw->nwm", Sp, A) if prob.mode == "uvw" else np.einsum("nqum,qu->num", Sp, A)


def _adjoint_state(prob, A, g):
    """S_bar[n, q, u, m_o] = m_bar A^T of one path (eq. receiver_adjoint)."""
    return np.einsum("quw,nwm->nqum", A, g) if prob.mode == "uvw" else np.einsum("qu,num->nqum", A, g)


def _state_T_mbar(prob, Sp, g):
    """A_bar = S^T m_bar of one path, flattened like its weights (eq. receiver_adjoint)."""
    if prob.mode == "uvw":
        return np.einsum("nqum,nwm->quw", Sp, g).reshape(prob.K, -1)
    return np.einsum("nqum,num->qu", Sp, g)


def _mix(prob, S, W, N):
    """m = S A per output group  (eqs. receiver_mixing / receiver_matrix_product)."""
    mb = [np.zeros((N, mul, 2 * l + 1)) for (mul, l, _p) in prob.irreps_out]
    for p, Sp in zip(prob.paths, S):
        mb[p["i_out"]] += _state_times_A(prob, Sp, _A(prob, W, p))
    return mb


def fwd_receiver(prob, x, evec, phi, W, rowptr, sender):
    xb, recv, send = _prepare(prob, x, rowptr, sender)
    N = len(rowptr) - 1
    Y = _sh.sh(prob.lmax, _f64(evec))
    S = _receiver_state(prob, _f64(phi), _edge_C(prob, xb, Y, send), recv, N)
    return _ir.blocks_to_flat(_mix(prob, S, _f64(W), N), prob.irreps_out, prob.layout)


def _edge_adjoints(prob, xb, Y, send, recv, phi, Sbar, N, extra=None):
    """Per-edge G = sum_q phi_q S_bar_i[q], phi_bar, Y_bar and x_bar from a receiver adjoint state."""
    E = len(send)
    nsh = (prob.lmax + 1) ** 2
    gphi = np.zeros((E, prob.K))
    gY = np.zeros((E, nsh))
    gxb = [np.zeros_like(b) for b in xb]
    Cs = _edge_C(prob, xb, Y, send)
    for p, c, Sb, Ct in zip(prob.paths, prob.coeffs, Sbar, Cs):
        Sbe = Sb[recv]                                          # [E, K, C_in, d_out]
        G = np.einsum("eq,equm->eum", phi, Sbe)
        gphi += np.einsum("equm,eum->eq", Sbe, Ct)
        M = _contract_y(c, _sh_slice(Y, p["l_sh"]))
        np.add.at(gxb[p["i_in"]], send, np.matmul(G, np.swapaxes(M, 1, 2)))
        P = np.matmul(np.swapaxes(xb[p["i_in"]][send], 1, 2), G)
        l = p["l_sh"]
        gY[:, l * l:(l + 1) ** 2] += np.einsum("ijk,eik->ej", c, P)
    return gphi, gY, gxb


def bwd_receiver(prob, x, evec, phi, W, rowptr, sender, gout):
    xb, recv, send = _prepare(prob, x, rowptr, sender)
    evec, phi, W = _f64(evec), _f64(phi), _f64(W)
    N = len(rowptr) - 1
    gb = _ir.flat_to_blocks(_f64(gout), prob.irreps_out, prob.layout)
    Y = _sh.sh(prob.lmax, evec)
    J = _sh.sh_jacobian(prob.lmax, evec)
    S = _receiver_state(prob, phi, _edge_C(prob, xb, Y, send), recv, N)
    Sbar, gW = [], np.zeros_like(W)
    for p, Sp in zip(prob.paths, S):
        A = _A(prob, W, p)
        g = gb[p["i_out"]]
        Sbar.append(_adjoint_state(prob, A, g))              # S_bar = m_bar A^T   (eq. receiver_adjoint)
        gW[:, p["w_off"]:p["w_off"] + p["n_w"]] = _state_T_mbar(prob, Sp, g)
    gphi, gY, gxb = _edge_adjoints(prob, xb, Y, send, recv, phi, Sbar, N)
    return dict(gx=_ir.blocks_to_flat(gxb, prob.irreps_in, prob.layout),
                gevec=np.einsum("ej,ejk->ek", gY, J), gphi=gphi, gW=gW)


def dbwd_receiver(prob, x, evec, phi, W, rowptr, sender, gout,
                  t_gx=None, t_gevec=None, t_gphi=None, t_gW=None):
    """Receiver-program form of dbwd (eq. receiver_double_adjoint, d m_bar = 0)."""
    xb, recv, send = _prepare(prob, x, rowptr, sender)
    evec, phi, W = _f64(evec), _f64(phi), _f64(W)
    N, E = len(rowptr) - 1, len(send)
    gb = _ir.flat_to_blocks(_f64(gout), prob.irreps_out, prob.layout)
    xdb = (_ir.flat_to_blocks(_f64(t_gx), prob.irreps_in, prob.layout)
           if t_gx is not None else [np.zeros_like(b) for b in xb])
    rdot = _f64(t_gevec) if t_gevec is not None else np.zeros((E, 3))
    phid = _f64(t_gphi) if t_gphi is not None else np.zeros((E, prob.K))
    Wd = _f64(t_gW) if t_gW is not None else np.zeros_like(W)
    Y = _sh.sh(prob.lmax, evec)
    J = _sh.sh_jacobian(prob.lmax, evec)
    Hs = _sh.sh_hessian(prob.lmax, evec)
    Yd = np.einsum("ejk,ek->ej", J, rdot)
    C = _edge_C(prob, xb, Y, send)
    Cd = [a + b for a, b in zip(_edge_C(prob, xdb, Y, send), _edge_C(prob, xb, Yd, send))]
    S = _receiver_state(prob, phi, C, recv, N)
    dS = [a + b for a, b in zip(_receiver_state(prob, phid, C, recv, N),
                                _receiver_state(prob, phi, Cd, recv, N))]
    m_dot = [a + b for a, b in zip(_mix(prob, dS, W, N), _mix(prob, S, Wd, N))]   # dm = dS A + S dA
    g_W = np.zeros_like(W)
    g_phi = np.zeros((E, prob.K))
    nsh = (prob.lmax + 1) ** 2
    gY = np.zeros((E, nsh))
    Ybar = np.zeros((E, nsh))
    g_xb = [np.zeros_like(b) for b in xb]
    for p, c, Ct, Ctd, dSp in zip(prob.paths, prob.coeffs, C, Cd, dS):
        A, Ad, g = _A(prob, W, p), _A(prob, Wd, p), gb[p["i_out"]]
        Sb = _adjoint_state(prob, A, g)[recv]                 # S_bar  = m_bar A^T
        Sbp = _adjoint_state(prob, Ad, g)[recv]               # S_bar' = m_bar dA^T
        g_W[:, p["w_off"]:p["w_off"] + p["n_w"]] = _state_T_mbar(prob, dSp, g)
        G = np.einsum("eq,equm->eum", phi, Sb)
        Gd = np.einsum("eq,equm->eum", phid, Sb) + np.einsum("eq,equm->eum", phi, Sbp)
        g_phi += np.einsum("equm,eum->eq", Sb, Ctd) + np.einsum("equm,eum->eq", Sbp, Ct)
        l = p["l_sh"]
        M = _contract_y(c, _sh_slice(Y, l))
        Md = _contract_y(c, _sh_slice(Yd, l))
        np.add.at(g_xb[p["i_in"]], send,
                  np.matmul(Gd, np.swapaxes(M, 1, 2)) + np.matmul(G, np.swapaxes(Md, 1, 2)))
        xs, xds = xb[p["i_in"]][send], xdb[p["i_in"]][send]
        Pd = np.matmul(np.swapaxes(xs, 1, 2), Gd) + np.matmul(np.swapaxes(xds, 1, 2), G)
        gY[:, l * l:(l + 1) ** 2] += np.einsum("ijk,eik->ej", c, Pd)
        P = np.matmul(np.swapaxes(xs, 1, 2), G)
        Ybar[:, l * l:(l + 1) ** 2] += np.einsum("ijk,eik->ej", c, P)
    g_evec = np.einsum("ej,ejk->ek", gY, J) + np.einsum("ej,ejkl,el->ek", Ybar, Hs, rdot)
    return dict(g_gout=_ir.blocks_to_flat(m_dot, prob.irreps_out, prob.layout),
                g_x=_ir.blocks_to_flat(g_xb, prob.irreps_in, prob.layout),
                g_evec=g_evec, g_phi=g_phi, g_W=g_W)
