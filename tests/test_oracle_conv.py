"""Pins for the oracle convolution: symmetry, special cases, derivatives, second route."""

import numpy as np
import pytest

from oracle import conv, irreps as ir, sh
from tests.test_oracle_cg import random_rotation, wigner_from_sh


def small_case(irr_in, lmax, irr_out, K, N, E, seed, empty_node=True):
    rng = np.random.default_rng(seed)
    prob = conv.Problem(irr_in, lmax, irr_out, K)
    recv = rng.integers(0, N - 1 if empty_node else N, E)  # node N-1 receives nothing
    send = rng.integers(0, N, E)
    order = np.lexsort((send, recv))
    recv, send = recv[order], send[order]
    rowptr = np.concatenate([[0], np.cumsum(np.bincount(recv, minlength=N))])
    return dict(prob=prob, rowptr=rowptr, sender=send, rng=rng,
                x=rng.normal(size=(N, prob.dim_in)), evec=rng.normal(size=(E, 3)),
                phi=rng.normal(size=(E, K)), W=rng.normal(size=(K, prob.n_w)),
                gout=rng.normal(size=(N, prob.dim_out)))


def args(c):
    return (c["prob"], c["x"], c["evec"], c["phi"], c["W"], c["rowptr"], c["sender"])


def block_transform(irreps, flat, R, layout="ir_mul"):
    """Apply the O(3) element R to a flat feature array (parity p: factor p^[det R < 0])."""
    det = np.linalg.det(R)
    Rp = R * np.sign(det)
    blocks = ir.flat_to_blocks(flat, irreps, layout)
    out = []
    for b, (mul, l, p) in zip(blocks, irreps):
        D = wigner_from_sh(l, Rp)
        f = p if det < 0 else 1
        out.append(f * np.einsum("ij,nuj->nui", D, b))
    return ir.blocks_to_flat(out, irreps, layout)


IRR = ("3x0e+2x1o+2x1e+2x2e+1x3o", 3, "2x0e+2x0o+3x1o+1x1e+2x2e+1x2o+1x3o")


@pytest.mark.parametrize("improper", [False, True])
def test_equivariance_o3(improper):
    c = small_case(*IRR, K=3, N=6, E=20, seed=1)
    rng = np.random.default_rng(11)
    R = random_rotation(rng)
    if improper:
        R = -R
    m = conv.fwd(*args(c))
    xr = block_transform(c["prob"].irreps_in, c["x"], R)
    mr = conv.fwd(c["prob"], xr, c["evec"] @ R.T, c["phi"], c["W"], c["rowptr"], c["sender"])
    np.testing.assert_allclose(mr, block_transform(c["prob"].irreps_out, m, R), atol=1e-10)


def test_parity_selection_catches_wrong_parity_path():
    # 1o x 1o -> 1e is allowed; 1o x 1o -> 1o is not, so an output 1o gets nothing from 1o x Y_1
    c = small_case("1x1o", 1, "1x1o+1x1e", K=2, N=4, E=10, seed=2)
    m = conv.fwd(*args(c))
    blocks = ir.flat_to_blocks(m, c["prob"].irreps_out)
    # 1o output only receives 1o x Y_0
    prob0 = conv.Problem("1x1o", 0, "1x1o+1x1e", 2)
    W0 = np.zeros((2, prob0.n_w))
    W0[:, :] = c["W"][:, :1]   # the 1o x 0e -> 1o path has offset 0 in both problems
    m0 = conv.fwd(prob0, c["x"], c["evec"], c["phi"], W0, c["rowptr"], c["sender"])
    np.testing.assert_allclose(blocks[0], ir.flat_to_blocks(m0, prob0.irreps_out)[0], atol=1e-12)


def test_scalar_case_is_weighted_spmm():
    # 0e x 0e -> 0e: m_i[w] = sum_e sum_u (phi_e A)[u, w] x_j[u]
    c = small_case("3x0e", 0, "2x0e", K=4, N=7, E=25, seed=3)
    m = conv.fwd(*args(c))
    recv = conv.receivers_from_rowptr(c["rowptr"])
    dense = np.zeros((7, 7, 4))     # adjacency weighted by phi: [recv, send, q]
    np.add.at(dense, (recv, c["sender"]), c["phi"])
    A = c["W"].reshape(4, 3, 2)
    ref = np.einsum("ijq,ju,quw->iw", dense, c["x"], A)
    np.testing.assert_allclose(m, ref, atol=1e-12)


def test_dot_cross_and_scaling_special_cases():
    rng = np.random.default_rng(4)
    N, E = 5, 12
    recv = np.sort(rng.integers(0, N, E))
    send = rng.integers(0, N, E)
    rowptr = np.concatenate([[0], np.cumsum(np.bincount(recv, minlength=N))])
    ev = rng.normal(size=(E, 3))
    rhat = ev / np.linalg.norm(ev, axis=1, keepdims=True)
    phi = np.ones((E, 1))
    # 1o x 1o -> 0e: x . rhat (CG = delta / sqrt3 and Y_1 = sqrt3 rhat in (y, z, x) order)
    p = conv.Problem("1x1o", 1, "1x0e", 1)
    x = rng.normal(size=(N, 3))          # (y, z, x) components
    m = conv.fwd(p, x, ev, phi, np.ones((1, 1)), rowptr, send)
    r_yzx = rhat[:, [1, 2, 0]]
    ref = np.zeros(N)
    np.add.at(ref, recv, (x[send] * r_yzx).sum(1))
    np.testing.assert_allclose(m[:, 0], ref, atol=1e-12)
    # 1o x 1o -> 1e: sqrt(3/2) x cross rhat in the (y, z, x) order
    p = conv.Problem("1x1o", 1, "1x1e", 1)
    m = conv.fwd(p, x, ev, phi, np.ones((1, 1)), rowptr, send)
    xs = x[send][:, [2, 0, 1]]          # back to (x, y, z)
    cr = np.cross(xs, rhat)[:, [1, 2, 0]]
    ref = np.zeros((N, 3))
    np.add.at(ref, recv, np.sqrt(1.5) * cr)
    np.testing.assert_allclose(m, ref, atol=1e-12)
    # 0e x 1o -> 1o: x_u Y_1
    p = conv.Problem("2x0e", 1, "1x1o", 1)
    x = rng.normal(size=(N, 2))
    W = np.array([[0.0, 0.0, 0.7, -0.3]])  # path order: (0e,0e->?) none; (0e, 1o -> 1o) has offset 0
    W = W[:, -p.n_w:]
    m = conv.fwd(p, x, ev, phi, W, rowptr, send)
    Y1 = sh.sh(1, ev)[:, 1:]
    ref = np.zeros((N, 3))
    np.add.at(ref, recv, (x[send] @ W.reshape(2, 1))[:, :1] * Y1)
    np.testing.assert_allclose(m, ref, atol=1e-12)


def test_linearity_and_scale_invariance():
    c = small_case(*IRR, K=3, N=6, E=20, seed=5)
    m = conv.fwd(*args(c))
    p, x, ev, phi, W, rp, s = args(c)
    np.testing.assert_allclose(conv.fwd(p, 2.5 * x, ev, phi, W, rp, s), 2.5 * m, atol=1e-11)
    np.testing.assert_allclose(conv.fwd(p, x, ev, -1.5 * phi, W, rp, s), -1.5 * m, atol=1e-11)
    np.testing.assert_allclose(conv.fwd(p, x, ev, phi, 0.5 * W, rp, s), 0.5 * m, atol=1e-11)
    np.testing.assert_allclose(conv.fwd(p, x, 3.0 * ev, phi, W, rp, s), m, atol=1e-11)


def test_empty_receiver_gets_zero():
    c = small_case(*IRR, K=3, N=6, E=20, seed=6, empty_node=True)
    assert c["rowptr"][-1] == c["rowptr"][-2]
    m = conv.fwd(*args(c))
    assert np.all(m[-1] == 0)


def test_edge_order_and_node_relabel_invariance():
    c = small_case(*IRR, K=3, N=6, E=20, seed=7)
    m = conv.fwd(*args(c))
    rng = np.random.default_rng(8)
    perm = rng.permutation(6)                  # new id of node i is perm[i]
    recv = conv.receivers_from_rowptr(c["rowptr"])
    nr, ns = perm[recv], perm[c["sender"]]
    order = np.lexsort((rng.random(len(nr)), nr))   # receiver-sorted, random order inside a receiver
    rowptr = np.concatenate([[0], np.cumsum(np.bincount(nr, minlength=6))])
    xp = np.empty_like(c["x"])
    xp[perm] = c["x"]
    m2 = conv.fwd(c["prob"], xp, c["evec"][order], c["phi"][order], c["W"], rowptr, ns[order])
    np.testing.assert_allclose(m2[perm], m, atol=1e-11)


def test_layouts_agree():
    c = small_case(*IRR, K=3, N=6, E=20, seed=9)
    m = conv.fwd(*args(c))
    p2 = conv.Problem(*IRR[:2], IRR[2], 3, layout="mul_ir")
    xb = ir.flat_to_blocks(c["x"], p2.irreps_in, "ir_mul")
    x2 = ir.blocks_to_flat(xb, p2.irreps_in, "mul_ir")
    m2 = conv.fwd(p2, x2, c["evec"], c["phi"], c["W"], c["rowptr"], c["sender"])
    for b2, b1 in zip(ir.flat_to_blocks(m2, p2.irreps_out, "mul_ir"), ir.flat_to_blocks(m, p2.irreps_out, "ir_mul")):
        np.testing.assert_allclose(b2, b1, atol=1e-12)


def fd_check(f, arrays, grads, rng, h=1e-5, rtol=1e-7):
    for i, g in enumerate(grads):
        if g is None:
            continue
        d = rng.normal(size=arrays[i].shape)
        a = list(arrays)
        a[i] = arrays[i] + h * d
        lp = f(*a)
        a[i] = arrays[i] - h * d
        lm = f(*a)
        fd = (lp - lm) / (2 * h)
        an = float((g * d).sum())
        assert abs(fd - an) <= rtol * max(1.0, abs(an)), (i, fd, an)


@pytest.mark.parametrize("norm", ["none", "fan_in"])
def test_backward_finite_differences(norm):
    c = small_case("2x0e+2x1o+1x2e", 2, "2x0e+1x1o+2x1e+1x2e", K=3, N=5, E=14, seed=10)
    prob = conv.Problem("2x0e+2x1o+1x2e", 2, "2x0e+1x1o+2x1e+1x2e", 3, normalization=norm)
    a = [c["x"], c["evec"], c["phi"], c["W"]]
    b = conv.bwd(prob, *a, c["rowptr"], c["sender"], c["gout"])

    def L(x, ev, phi, W):
        return float((c["gout"] * conv.fwd(prob, x, ev, phi, W, c["rowptr"], c["sender"])).sum())
    fd_check(L, a, [b["gx"], b["gevec"], b["gphi"], b["gW"]], np.random.default_rng(0))
    # degree-0 homogeneity of Y in evec: <evec_bar_e, evec_e> = 0
    np.testing.assert_allclose((b["gevec"] * c["evec"]).sum(1), 0, atol=1e-11)


@pytest.mark.parametrize("active", ["all", "evec"])
def test_double_backward_finite_differences(active):
    c = small_case("2x0e+2x1o+1x2e", 2, "2x0e+1x1o+2x1e+1x2e", K=3, N=5, E=14, seed=11)
    prob = c["prob"]
    rng = c["rng"]
    t = dict(x=rng.normal(size=c["x"].shape), evec=rng.normal(size=c["evec"].shape),
             phi=rng.normal(size=c["phi"].shape), W=rng.normal(size=c["W"].shape))
    if active == "evec":
        t = dict(x=None, evec=t["evec"], phi=None, W=None)
    d = conv.dbwd(prob, c["x"], c["evec"], c["phi"], c["W"], c["rowptr"], c["sender"], c["gout"],
                  t_gx=t["x"], t_gevec=t["evec"], t_gphi=t["phi"], t_gW=t["W"])

    def L2(x, ev, phi, W, g):
        b = conv.bwd(prob, x, ev, phi, W, c["rowptr"], c["sender"], g)
        return float(sum((b[k] * t[n]).sum() for k, n in
                         (("gx", "x"), ("gevec", "evec"), ("gphi", "phi"), ("gW", "W")) if t[n] is not None))
    a = [c["x"], c["evec"], c["phi"], c["W"], c["gout"]]
    fd_check(L2, a, [d["g_x"], d["g_evec"], d["g_phi"], d["g_W"], d["g_gout"]], np.random.default_rng(1))


def test_receiver_route_matches_materialised():
    c = small_case(*IRR, K=3, N=6, E=20, seed=12)
    a = args(c)
    m1, m2 = conv.fwd(*a), conv.fwd_receiver(*a)
    np.testing.assert_allclose(m2, m1, rtol=0, atol=1e-12 * np.abs(m1).max())
    b1, b2 = conv.bwd(*a, c["gout"]), conv.bwd_receiver(*a, c["gout"])
    for k in b1:
        np.testing.assert_allclose(b2[k], b1[k], rtol=0, atol=1e-12 * np.abs(b1[k]).max())
    rng = c["rng"]
    t = dict(t_gx=rng.normal(size=c["x"].shape), t_gevec=rng.normal(size=c["evec"].shape),
             t_gphi=rng.normal(size=c["phi"].shape), t_gW=rng.normal(size=c["W"].shape))
    d1, d2 = conv.dbwd(*a, c["gout"], **t), conv.dbwd_receiver(*a, c["gout"], **t)
    for k in d1:
        np.testing.assert_allclose(d2[k], d1[k], rtol=0, atol=1e-12 * np.abs(d1[k]).max())
