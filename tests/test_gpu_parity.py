"""GPU parity: the HIP library (through its C ABI) against the float64 oracle.

Each case runs fwd, bwd and dbwd through libsobek_hip and compares every
output element-wise with the oracle on the same seeded inputs, using the
max-norm relative error ||gpu - oracle||_inf / ||oracle||_inf with the
tolerances 1e-4 (fp32 forward) and 5e-4 (fp32 backward and double backward).
Graphs are small enough for the oracle to finish in seconds but span several
receiver chunks, GEMM tiles and a ragged tail.
"""

import numpy as np
import pytest

from oracle import conv as oc
from tests.cases import BWD_TOL, FWD_TOL, make_case, max_rel

pytestmark = pytest.mark.gpu


def _t(a, dev="cuda"):
    import torch
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def _n(t):
    return None if t is None else t.detach().cpu().numpy()


def setup(case, layout="ir_mul", normalization="none"):
    import torch  # noqa: F401
    from paper_2607_18074_amd import api
    irr_in, lmax, irr_out, K = case["sig"]
    plan = api.Plan(irr_in, lmax, irr_out, K, layout=layout, normalization=normalization)
    g = case["graph"]
    graph = api.Graph(_t(g.rowptr), _t(g.sender))
    prob = oc.Problem(irr_in, lmax, irr_out, K, normalization=normalization, layout=layout)
    return api, plan, graph, prob


def oracle_args(case, prob):
    g = case["graph"]
    return (prob, case["x"], g.evec, g.phi, case["W"], g.rowptr, g.sender)


CASES = [
    ("tiny", 64, 1024, 0, 0),
    ("small", 300, 4000, 1, 3),
    ("medium", 120, 1500, 2, 2),
    ("wide", 60, 600, 3, 1),
    ("odd", 50, 700, 4, 2),
    ("widec", 70, 800, 5, 1),
]


@pytest.mark.parametrize("sig,N,E,seed,iso", CASES)
def test_forward(gpu, sig, N, E, seed, iso):
    case = make_case(sig, N, E, seed, isolated=iso)
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    out = api.conv_fwd(plan, graph, _t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    ref = oc.fwd(*oracle_args(case, prob))
    err = max_rel(_n(out), ref)
    print(f"fwd {sig}: max rel err {err:.2e}")
    assert err <= FWD_TOL
    if iso:
        assert np.all(_n(out)[-iso:] == 0)


@pytest.mark.parametrize("sig,N,E,seed,iso", CASES)
def test_backward(gpu, sig, N, E, seed, iso):
    case = make_case(sig, N, E, seed, isolated=iso)
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    outs = api.conv_bwd(plan, graph, _t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]), _t(case["gout"]))
    ref = oc.bwd(*oracle_args(case, prob), case["gout"])
    for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
        err = max_rel(_n(o), ref[name])
        print(f"bwd {sig} {name}: max rel err {err:.2e}")
        assert err <= BWD_TOL, name


@pytest.mark.parametrize("active", ["all", "evec", "x_phi", "W"])
@pytest.mark.parametrize("sig,N,E,seed,iso", CASES)
def test_double_backward(gpu, sig, N, E, seed, iso, active):
    case = make_case(sig, N, E, seed, isolated=iso)
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    keep = dict(all=("x", "evec", "phi", "W"), evec=("evec",), x_phi=("x", "phi"), W=("W",))[active]
    t = {k: (v if k in keep else None) for k, v in case["cot"].items()}
    outs = api.conv_dbwd(plan, graph, _t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]), _t(case["gout"]),
                         _t(t["x"]), _t(t["evec"]), _t(t["phi"]), _t(t["W"]))
    ref = oc.dbwd(*oracle_args(case, prob), case["gout"], t_gx=t["x"], t_gevec=t["evec"], t_gphi=t["phi"],
                  t_gW=t["W"])
    for name, o in zip(("g_gout", "g_x", "g_evec", "g_phi", "g_W"), outs):
        r = ref[name]
        if np.abs(r).max() == 0:
            assert np.abs(_n(o)).max() == 0, name
            continue
        err = max_rel(_n(o), r)
        print(f"dbwd {sig} [{active}] {name}: max rel err {err:.2e}")
        assert err <= BWD_TOL, name


def test_deterministic_and_chunk_invariant(gpu):
    case = make_case("small", 400, 6000, 7, isolated=1)
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    gout = _t(case["gout"])
    a = [_n(api.conv_fwd(plan, graph, *args))] + [_n(o) for o in api.conv_bwd(plan, graph, *args, gout)]
    b = [_n(api.conv_fwd(plan, graph, *args))] + [_n(o) for o in api.conv_bwd(plan, graph, *args, gout)]
    for u, v in zip(a, b):
        assert np.array_equal(u, v)          # bitwise run-to-run determinism
    # a small budget forces many receiver chunks; results stay within tolerance
    c = [_n(api.conv_fwd(plan, graph, *args, budget=1 << 20))] + \
        [_n(o) for o in api.conv_bwd(plan, graph, *args, gout, budget=1 << 20)]
    ref = oc.bwd(*oracle_args(case, prob), case["gout"])
    assert max_rel(c[0], oc.fwd(*oracle_args(case, prob))) <= FWD_TOL
    for name, o in zip(("gx", "gevec", "gphi", "gW"), c[1:]):
        assert max_rel(o, ref[name]) <= BWD_TOL, name


@pytest.mark.parametrize("layout,norm", [("mul_ir", "none"), ("ir_mul", "fan_in"), ("mul_ir", "fan_in")])
def test_layout_and_normalisation(gpu, layout, norm):
    case = make_case("odd", 40, 500, 8, isolated=1)
    from oracle import irreps as ir
    api, plan, graph, prob = setup(case, layout=layout, normalization=norm)
    g = case["graph"]
    irr_in, irr_out = prob.irreps_in, prob.irreps_out
    x = ir.blocks_to_flat(ir.flat_to_blocks(case["x"], irr_in, "ir_mul"), irr_in, layout).astype(np.float32)
    gout = ir.blocks_to_flat(ir.flat_to_blocks(case["gout"], irr_out, "ir_mul"), irr_out, layout).astype(np.float32)
    tx = ir.blocks_to_flat(ir.flat_to_blocks(case["cot"]["x"], irr_in, "ir_mul"), irr_in, layout).astype(np.float32)
    oa = (prob, x, g.evec, g.phi, case["W"], g.rowptr, g.sender)
    out = api.conv_fwd(plan, graph, _t(x), _t(g.evec), _t(g.phi), _t(case["W"]))
    assert max_rel(_n(out), oc.fwd(*oa)) <= FWD_TOL
    outs = api.conv_bwd(plan, graph, _t(x), _t(g.evec), _t(g.phi), _t(case["W"]), _t(gout))
    ref = oc.bwd(*oa, gout)
    for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
        assert max_rel(_n(o), ref[name]) <= BWD_TOL, name
    c = case["cot"]
    outs = api.conv_dbwd(plan, graph, _t(x), _t(g.evec), _t(g.phi), _t(case["W"]), _t(gout), _t(tx),
                         _t(c["evec"]), _t(c["phi"]), _t(c["W"]))
    ref = oc.dbwd(*oa, gout, t_gx=tx, t_gevec=c["evec"], t_gphi=c["phi"], t_gW=c["W"])
    for name, o in zip(("g_gout", "g_x", "g_evec", "g_phi", "g_W"), outs):
        assert max_rel(_n(o), ref[name]) <= BWD_TOL, name


def test_empty_graph(gpu):
    import torch
    from paper_2607_18074_amd import api
    plan = api.Plan("4x0e+2x1o", 1, "3x0e+2x1o", 4)
    N = 5
    graph = api.Graph(torch.zeros(N + 1, dtype=torch.int32, device="cuda"), torch.zeros(0, dtype=torch.int32,
                                                                                         device="cuda"))
    x = torch.randn(N, plan.dim_in, device="cuda")
    ev = torch.zeros(0, 3, device="cuda")
    ph = torch.zeros(0, 4, device="cuda")
    W = torch.randn(4, plan.n_weights, device="cuda")
    out = api.conv_fwd(plan, graph, x, ev, ph, W)
    assert torch.all(out == 0)
    gx, gev, gph, gW = api.conv_bwd(plan, graph, x, ev, ph, W, torch.randn(N, plan.dim_out, device="cuda"))
    assert torch.all(gx == 0) and torch.all(gW == 0)


def test_autograd_matches_oracle(gpu):
    import torch
    case = make_case("small", 80, 900, 9)
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    x = _t(case["x"]).requires_grad_()
    ev = _t(g.evec).requires_grad_()
    ph = _t(g.phi).requires_grad_()
    W = _t(case["W"]).requires_grad_()
    m = api.tp_conv(plan, graph, x, ev, ph, W)
    gout = _t(case["gout"])
    gx, gev, gph, gW = torch.autograd.grad(m, (x, ev, ph, W), gout, create_graph=True)
    ref = oc.bwd(*oracle_args(case, prob), case["gout"])
    assert max_rel(_n(gev), ref["gevec"]) <= BWD_TOL
    # L2 = sum |g_evec|^2: its gradients are the double backward with t_gevec = 2 g_evec
    L2 = (gev ** 2).sum()
    d = torch.autograd.grad(L2, (x, ev, ph, W))
    r = oc.dbwd(*oracle_args(case, prob), case["gout"], t_gevec=2 * _n(gev).astype(np.float64))
    for name, o in zip(("g_x", "g_evec", "g_phi", "g_W"), d):
        assert max_rel(_n(o), r[name]) <= BWD_TOL, name


@pytest.mark.parametrize("sig,N,E,seed", [("small", 300, 4000, 11), ("odd", 50, 700, 12), ("medium", 120, 1500, 13)])
def test_retained_state(gpu, sig, N, E, seed):
    """Forward that keeps S, and the backward that reads it, against the oracle and the recomputing path."""
    import torch
    case = make_case(sig, N, E, seed, isolated=2)
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    state = api.new_state(plan, graph)
    state.fill_(float("nan"))                       # every element the backward reads must be written
    m = api.conv_fwd(plan, graph, *args, state=state, budget=1 << 20)   # small budget: the state is one chunk anyway
    assert max_rel(_n(m), oc.fwd(*oracle_args(case, prob))) <= FWD_TOL
    # the state GEMM's split-K depends on the chunk size, so budgets differ only in summation order
    assert max_rel(_n(m), _n(api.conv_fwd(plan, graph, *args))) <= 1e-5
    gout = _t(case["gout"])
    ref = oc.bwd(*oracle_args(case, prob), case["gout"])
    for budget in (0, 1 << 20):                     # one chunk, and many chunks for the edge stage
        outs = api.conv_bwd(plan, graph, *args, gout, state=state, budget=budget)
        for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
            err = max_rel(_n(o), ref[name])
            print(f"bwd (retained S, budget {budget}) {sig} {name}: max rel err {err:.2e}")
            assert err <= BWD_TOL, name
    # the adjoint state kept by the backward serves the double backward (all four cotangents and edge-only)
    adj = api.new_state(plan, graph)
    adj.fill_(float("nan"))
    outs = api.conv_bwd(plan, graph, *args, gout, state=state, adj_state=adj)
    for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
        assert max_rel(_n(o), ref[name]) <= BWD_TOL, name
    c = case["cot"]
    for keep in (("x", "evec", "phi", "W"), ("evec",)):
        t = {k: (v if k in keep else None) for k, v in c.items()}
        for budget in (0, 1 << 20):
            outs = api.conv_dbwd(plan, graph, *args, gout, _t(t["x"]), _t(t["evec"]), _t(t["phi"]), _t(t["W"]),
                                 adj_state=adj, budget=budget)
            r = oc.dbwd(*oracle_args(case, prob), case["gout"], t_gx=t["x"], t_gevec=t["evec"], t_gphi=t["phi"],
                        t_gW=t["W"])
            for name, o in zip(("g_gout", "g_x", "g_evec", "g_phi", "g_W"), outs):
                if np.abs(r[name]).max() == 0:
                    assert np.abs(_n(o)).max() == 0, name
                    continue
                err = max_rel(_n(o), r[name])
                print(f"dbwd (kept Sbar, {keep}, budget {budget}) {sig} {name}: max rel err {err:.2e}")
                assert err <= BWD_TOL, name
    # W does not enter S: a state kept with other weights serves as well
    m2 = api.conv_fwd(plan, graph, args[0], args[1], args[2], 2 * args[3], state=state)
    torch.cuda.synchronize()
    assert torch.isfinite(m2).all()
    outs = api.conv_bwd(plan, graph, *args, gout, state=state)
    assert max_rel(_n(outs[3]), ref["gW"]) <= BWD_TOL


def test_autograd_retained_state(gpu):
    import torch
    case = make_case("small", 80, 900, 14)
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    x = _t(case["x"]).requires_grad_()
    ev = _t(g.evec).requires_grad_()
    ph = _t(g.phi).requires_grad_()
    W = _t(case["W"]).requires_grad_()
    m = api.tp_conv(plan, graph, x, ev, ph, W, retain_state=True)
    gx, gev, gph, gW = torch.autograd.grad(m, (x, ev, ph, W), _t(case["gout"]), create_graph=True)
    ref = oc.bwd(*oracle_args(case, prob), case["gout"])
    for name, o in zip(("gx", "gevec", "gphi", "gW"), (gx, gev, gph, gW)):
        assert max_rel(_n(o), ref[name]) <= BWD_TOL, name
    d = torch.autograd.grad((gev ** 2).sum(), (x, ev, ph, W))
    r = oc.dbwd(*oracle_args(case, prob), case["gout"], t_gevec=2 * _n(gev).astype(np.float64))
    for name, o in zip(("g_x", "g_evec", "g_phi", "g_W"), d):
        assert max_rel(_n(o), r[name]) <= BWD_TOL, name


def test_kept_states_chunk_by_edges_only(gpu):
    """With S and Sbar both kept the backward needs no per-receiver workspace: its chunks are bounded by the
    per-edge x-gradient contributions alone (a regression test for chunks of one receiver each)."""
    from paper_2607_18074_amd import _lib
    case = make_case("small", 300, 4000, 15)
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    state, adj = api.new_state(plan, graph), api.new_state(plan, graph)
    api.conv_fwd(plan, graph, *args, state=state)
    budget = 2 << 20      # contributions of 4000 edges x 288 floats = 4.6 MB: a few chunks
    ws = graph.workspace(plan, "bwd", budget)
    _lib.profile_reset()
    _lib.profile_enable(True)
    outs = api.conv_bwd(plan, graph, *args, _t(case["gout"]), state=state, adj_state=adj, ws=ws)
    prof = _lib.profile_read()
    _lib.profile_enable(False)
    n_edge = prof["sobek_bwd_E"][0]
    print("bwd_E launches", n_edge, "workspace", ws.numel())
    assert 2 <= n_edge <= 10
    ref = oc.bwd(*oracle_args(case, prob), case["gout"])
    for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
        assert max_rel(_n(o), ref[name]) <= BWD_TOL, name


def test_windows_split_high_degree_receivers(gpu):
    """A budget whose edge windows are shorter than a receiver's in-degree: receivers are split across
    windows, and inside a window their edges are spread over blockIdx.y; backward and double backward
    still match the oracle."""
    from paper_2607_18074_amd import _lib
    case = make_case("small", 40, 8000, 16)        # mean in-degree 200
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    budget = 3 << 19                                  # 1.5 MiB: windows of a few hundred edges
    _lib.profile_reset()
    _lib.profile_enable(True)
    outs = api.conv_bwd(plan, graph, *args, _t(case["gout"]), budget=budget)
    prof = _lib.profile_read()
    _lib.profile_enable(False)
    print("bwd_E launches", prof["sobek_bwd_E"][0], "receivers", g.N, "edges", g.E)
    assert prof["sobek_bwd_E"][0] >= 4
    ref = oc.bwd(*oracle_args(case, prob), case["gout"])
    for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
        assert max_rel(_n(o), ref[name]) <= BWD_TOL, name
    cot = case["cot"]
    dref = oc.dbwd(*oracle_args(case, prob), case["gout"], t_gx=cot["x"], t_gevec=cot["evec"], t_gphi=cot["phi"],
                   t_gW=cot["W"])
    outs = api.conv_dbwd(plan, graph, *args, _t(case["gout"]), _t(cot["x"]), _t(cot["evec"]), _t(cot["phi"]),
                         _t(cot["W"]), budget=budget)
    for name, o in zip(("g_gout", "g_x", "g_evec", "g_phi", "g_W"), outs):
        assert max_rel(_n(o), dref[name]) <= BWD_TOL, name
