"""Pins for the channelwise (uvu) oracle, eq. uvu_connection.

A channelwise path is a fully connected one whose C_in x C_out weight block is
diagonal: W_uvw[q, u, w] = delta_uw W_uvu[q, u].  The uvw oracle (pinned by its
own tests) run on that embedding must give the same forward, the same node and
edge gradients, and a weight gradient whose diagonal is the uvu one; the uvu
code computes all of this with elementwise channel products instead of
matrices.  Finite differences, O(3) equivariance and the receiver route pin the
uvu derivatives independently.
"""

import numpy as np
import pytest

from oracle import cg, conv, irreps as ir
from tests.test_oracle_conv import block_transform, fd_check
from tests.test_oracle_cg import random_rotation

SIG = ("3x0e+3x1o+3x1e+3x2e", 2, "3x0e+3x1o+3x1e+3x2e")


def graph(N, E, rng, empty_node=True):
    recv = rng.integers(0, N - 1 if empty_node else N, E)
    send = rng.integers(0, N, E)
    order = np.lexsort((send, recv))
    recv, send = recv[order], send[order]
    return np.concatenate([[0], np.cumsum(np.bincount(recv, minlength=N))]), send


def embed(pu, pw, Wu):
    """Diagonal uvw weights [K, N_w(uvw)] holding the uvu weights [K, N_w(uvu)]."""
    Ww = np.zeros((Wu.shape[0], pw.n_w))
    for a, b in zip(pu.paths, pw.paths):
        C = a["c_in"]
        blk = Ww[:, b["w_off"]:b["w_off"] + b["n_w"]].reshape(-1, C, C)
        blk[:, np.arange(C), np.arange(C)] = Wu[:, a["w_off"]:a["w_off"] + a["n_w"]]
    return Ww


def diagonal(pu, pw, Gw):
    """uvu-shaped diagonal of a uvw-shaped weight gradient."""
    Gu = np.zeros((Gw.shape[0], pu.n_w))
    for a, b in zip(pu.paths, pw.paths):
        C = a["c_in"]
        blk = Gw[:, b["w_off"]:b["w_off"] + b["n_w"]].reshape(-1, C, C)
        Gu[:, a["w_off"]:a["w_off"] + a["n_w"]] = blk[:, np.arange(C), np.arange(C)]
    return Gu


def case(seed, K=3, N=7, E=24, sig=SIG):
    rng = np.random.default_rng(seed)
    pu = conv.Problem(*sig, K, mode="uvu")
    pw = conv.Problem(*sig, K, mode="uvw")
    rowptr, send = graph(N, E, rng)
    return dict(pu=pu, pw=pw, rowptr=rowptr, sender=send, rng=rng,
                x=rng.normal(size=(N, pu.dim_in)), evec=rng.normal(size=(E, 3)), phi=rng.normal(size=(E, K)),
                W=rng.normal(size=(K, pu.n_w)), gout=rng.normal(size=(N, pu.dim_out)))


def test_weight_counts_and_layout():
    c = case(0)
    pu, pw = c["pu"], c["pw"]
    assert [p["n_w"] for p in pu.paths] == [p["c_in"] for p in pu.paths]
    assert [p["n_w"] for p in pw.paths] == [p["c_in"] * p["c_out"] for p in pw.paths]
    assert pu.n_w == sum(p["c_in"] for p in pu.paths)
    assert [p["w_off"] for p in pu.paths] == list(np.cumsum([0] + [p["n_w"] for p in pu.paths])[:-1])


def test_unequal_multiplicities_rejected():
    with pytest.raises(ValueError):
        conv.Problem("4x0e+2x1o", 1, "4x0e+3x1o", 2, mode="uvu")


def test_fan_in_counts_paths():
    # an output irrep reached by n paths gets alpha = 1/sqrt(n) channelwise, 1/sqrt(sum C_in) fully connected
    paths = ir.enumerate_paths(ir.parse_irreps("2x0e+2x1o"), ir.sh_irreps(1), ir.parse_irreps("2x0e+2x1o"), "uvu")
    cu = cg.path_coefficients(paths, "fan_in", "uvu")
    cw = cg.path_coefficients(paths, "fan_in", "uvw")
    c0 = cg.path_coefficients(paths, "none", "uvu")
    for p, a, b, z in zip(paths, cu, cw, c0):
        n = sum(1 for q in paths if q["i_out"] == p["i_out"])
        s = sum(q["c_in"] for q in paths if q["i_out"] == p["i_out"])
        np.testing.assert_allclose(a, z / np.sqrt(n), atol=1e-15)
        np.testing.assert_allclose(b, z / np.sqrt(s), atol=1e-15)


def test_forward_and_backward_equal_diagonal_uvw():
    c = case(1)
    pu, pw = c["pu"], c["pw"]
    Ww = embed(pu, pw, c["W"])
    g = (c["x"], c["evec"], c["phi"])
    m_u = conv.fwd(pu, *g, c["W"], c["rowptr"], c["sender"])
    m_w = conv.fwd(pw, *g, Ww, c["rowptr"], c["sender"])
    np.testing.assert_allclose(m_u, m_w, rtol=0, atol=1e-12 * np.abs(m_w).max())
    b_u = conv.bwd(pu, *g, c["W"], c["rowptr"], c["sender"], c["gout"])
    b_w = conv.bwd(pw, *g, Ww, c["rowptr"], c["sender"], c["gout"])
    for k in ("gx", "gevec", "gphi"):
        np.testing.assert_allclose(b_u[k], b_w[k], rtol=0, atol=1e-12 * np.abs(b_w[k]).max())
    np.testing.assert_allclose(b_u["gW"], diagonal(pu, pw, b_w["gW"]), rtol=0, atol=1e-12 * np.abs(b_w["gW"]).max())


def test_double_backward_equals_diagonal_uvw():
    c = case(2)
    pu, pw, rng = c["pu"], c["pw"], c["rng"]
    Ww = embed(pu, pw, c["W"])
    tW = rng.normal(size=c["W"].shape)
    t = dict(t_gx=rng.normal(size=c["x"].shape), t_gevec=rng.normal(size=c["evec"].shape),
             t_gphi=rng.normal(size=c["phi"].shape))
    g = (c["x"], c["evec"], c["phi"])
    d_u = conv.dbwd(pu, *g, c["W"], c["rowptr"], c["sender"], c["gout"], t_gW=tW, **t)
    d_w = conv.dbwd(pw, *g, Ww, c["rowptr"], c["sender"], c["gout"], t_gW=embed(pu, pw, tW), **t)
    for k in ("g_gout", "g_x", "g_evec", "g_phi"):
        np.testing.assert_allclose(d_u[k], d_w[k], rtol=0, atol=1e-12 * np.abs(d_w[k]).max())
    np.testing.assert_allclose(d_u["g_W"], diagonal(pu, pw, d_w["g_W"]), rtol=0,
                               atol=1e-12 * np.abs(d_w["g_W"]).max())


def test_backward_finite_differences():
    c = case(3, K=2, N=5, E=12, sig=("2x0e+2x1o+2x2e", 2, "2x0e+2x1o+2x2e"))
    pu = c["pu"]
    a = [c["x"], c["evec"], c["phi"], c["W"]]
    b = conv.bwd(pu, *a, c["rowptr"], c["sender"], c["gout"])

    def L(x, ev, phi, W):
        return float((c["gout"] * conv.fwd(pu, x, ev, phi, W, c["rowptr"], c["sender"])).sum())
    fd_check(L, a, [b["gx"], b["gevec"], b["gphi"], b["gW"]], np.random.default_rng(0))


def test_double_backward_finite_differences():
    c = case(4, K=2, N=5, E=12, sig=("2x0e+2x1o+2x2e", 2, "2x0e+2x1o+2x2e"))
    pu, rng = c["pu"], c["rng"]
    t = dict(x=rng.normal(size=c["x"].shape), evec=rng.normal(size=c["evec"].shape),
             phi=rng.normal(size=c["phi"].shape), W=rng.normal(size=c["W"].shape))
    d = conv.dbwd(pu, c["x"], c["evec"], c["phi"], c["W"], c["rowptr"], c["sender"], c["gout"],
                  t_gx=t["x"], t_gevec=t["evec"], t_gphi=t["phi"], t_gW=t["W"])

    def L2(x, ev, phi, W, g):
        b = conv.bwd(pu, x, ev, phi, W, c["rowptr"], c["sender"], g)
        return float(sum((b[k] * t[n]).sum() for k, n in (("gx", "x"), ("gevec", "evec"), ("gphi", "phi"),
                                                          ("gW", "W"))))
    a = [c["x"], c["evec"], c["phi"], c["W"], c["gout"]]
    fd_check(L2, a, [d["g_x"], d["g_evec"], d["g_phi"], d["g_W"], d["g_gout"]], np.random.default_rng(1))


@pytest.mark.parametrize("improper", [False, True])
def test_equivariance_o3(improper):
    c = case(5, sig=("2x0e+2x1o+2x1e+2x2e+2x3o", 3, "2x0e+2x1o+2x1e+2x2e+2x3o"))
    pu = c["pu"]
    R = random_rotation(np.random.default_rng(12))
    if improper:
        R = -R
    m = conv.fwd(pu, c["x"], c["evec"], c["phi"], c["W"], c["rowptr"], c["sender"])
    xr = block_transform(pu.irreps_in, c["x"], R)
    mr = conv.fwd(pu, xr, c["evec"] @ R.T, c["phi"], c["W"], c["rowptr"], c["sender"])
    np.testing.assert_allclose(mr, block_transform(pu.irreps_out, m, R), atol=1e-10)


def test_receiver_route_matches_materialised():
    c = case(6)
    pu, rng = c["pu"], c["rng"]
    a = (pu, c["x"], c["evec"], c["phi"], c["W"], c["rowptr"], c["sender"])
    m1, m2 = conv.fwd(*a), conv.fwd_receiver(*a)
    np.testing.assert_allclose(m2, m1, rtol=0, atol=1e-12 * np.abs(m1).max())
    b1, b2 = conv.bwd(*a, c["gout"]), conv.bwd_receiver(*a, c["gout"])
    for k in b1:
        np.testing.assert_allclose(b2[k], b1[k], rtol=0, atol=1e-12 * np.abs(b1[k]).max())
    t = dict(t_gx=rng.normal(size=c["x"].shape), t_gevec=rng.normal(size=c["evec"].shape),
             t_gphi=rng.normal(size=c["phi"].shape), t_gW=rng.normal(size=c["W"].shape))
    d1, d2 = conv.dbwd(*a, c["gout"], **t), conv.dbwd_receiver(*a, c["gout"], **t)
    for k in d1:
        np.testing.assert_allclose(d2[k], d1[k], rtol=0, atol=1e-12 * np.abs(d1[k]).max())
