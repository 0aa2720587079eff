"""GPU parity of the channelwise (uvu) mode, eq. uvu_connection: forward, backward and double backward
through the C ABI against the float64 oracle, on one receiver chunk and on many (small workspace), with
and without retained receiver states, and through the autograd wrapper.  Tolerances as for uvw."""

import numpy as np
import pytest

from oracle import conv as oc
from tests.cases import BWD_TOL, FWD_TOL, make_case, max_rel

pytestmark = pytest.mark.gpu

CASES = [("uvu_small", 200, 3000, 21, 2), ("uvu_l3", 60, 700, 22, 1), ("uvu_odd", 50, 600, 23, 1),
         ("uvu_wide", 80, 1000, 26, 1), ("uvu_dead", 60, 700, 28, 1)]


def _t(a):
    import torch
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _n(t):
    return None if t is None else t.detach().cpu().numpy()


def setup(case):
    from paper_2607_18074_amd import api
    irr_in, lmax, irr_out, K = case["sig"]
    plan = api.Plan(irr_in, lmax, irr_out, K, mode="uvu")
    g = case["graph"]
    graph = api.Graph(_t(g.rowptr), _t(g.sender))
    prob = oc.Problem(irr_in, lmax, irr_out, K, mode="uvu")
    assert plan.n_weights == prob.n_w
    return api, plan, graph, prob


def oargs(case, prob):
    g = case["graph"]
    return (prob, case["x"], g.evec, g.phi, case["W"], g.rowptr, g.sender)


@pytest.mark.parametrize("sig,N,E,seed,iso", CASES)
@pytest.mark.parametrize("budget", [0, 1 << 20])
def test_uvu_fwd_bwd(gpu, sig, N, E, seed, iso, budget):
    case = make_case(sig, N, E, seed, isolated=iso, mode="uvu")
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    out = api.conv_fwd(plan, graph, *args, budget=budget)
    err = max_rel(_n(out), oc.fwd(*oargs(case, prob)))
    print(f"uvu fwd {sig} budget {budget}: {err:.2e}")
    assert err <= FWD_TOL
    ref = oc.bwd(*oargs(case, prob), case["gout"])
    outs = api.conv_bwd(plan, graph, *args, _t(case["gout"]), budget=budget)
    for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
        err = max_rel(_n(o), ref[name])
        print(f"uvu bwd {sig} budget {budget} {name}: {err:.2e}")
        assert err <= BWD_TOL, name


@pytest.mark.parametrize("sig,N,E,seed,iso", CASES)
@pytest.mark.parametrize("active", ["all", "evec"])
def test_uvu_dbwd(gpu, sig, N, E, seed, iso, active):
    case = make_case(sig, N, E, seed + 100, isolated=iso, mode="uvu")
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    cot = dict(case["cot"])
    if active == "evec":
        cot = dict(x=None, evec=cot["evec"], phi=None, W=None)
    ref = oc.dbwd(*oargs(case, prob), case["gout"], t_gx=cot["x"], t_gevec=cot["evec"], t_gphi=cot["phi"],
                  t_gW=cot["W"])
    for budget in (0, 1 << 20):
        outs = api.conv_dbwd(plan, graph, _t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]), _t(case["gout"]),
                             _t(cot["x"]), _t(cot["evec"]), _t(cot["phi"]), _t(cot["W"]), budget=budget)
        for name, o in zip(("g_gout", "g_x", "g_evec", "g_phi", "g_W"), outs):
            r = ref[name]
            if np.abs(r).max() == 0:
                assert np.abs(_n(o)).max() == 0, name
                continue
            err = max_rel(_n(o), r)
            print(f"uvu dbwd {sig} [{active}] budget {budget} {name}: {err:.2e}")
            assert err <= BWD_TOL, name


def test_uvu_retained_states(gpu):
    case = make_case("uvu_small", 150, 2000, 24, isolated=1, mode="uvu")
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    state, adj = api.new_state(plan, graph), api.new_state(plan, graph)
    m = api.conv_fwd(plan, graph, *args, state=state)
    assert max_rel(_n(m), oc.fwd(*oargs(case, prob))) <= FWD_TOL
    ref = oc.bwd(*oargs(case, prob), case["gout"])
    outs = api.conv_bwd(plan, graph, *args, _t(case["gout"]), state=state, adj_state=adj)
    for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
        assert max_rel(_n(o), ref[name]) <= BWD_TOL, name
    cot = case["cot"]
    dref = oc.dbwd(*oargs(case, prob), case["gout"], t_gevec=cot["evec"], t_gW=cot["W"])
    outs = api.conv_dbwd(plan, graph, *args, _t(case["gout"]), t_gevec=_t(cot["evec"]), t_gW=_t(cot["W"]),
                         adj_state=adj)
    for name, o in zip(("g_gout", "g_x", "g_evec", "g_phi", "g_W"), outs):
        assert max_rel(_n(o), dref[name]) <= BWD_TOL, name


def test_uvu_autograd(gpu):
    import torch
    case = make_case("uvu_small", 80, 900, 25, mode="uvu")
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    x = _t(case["x"]).requires_grad_()
    ev = _t(g.evec).requires_grad_()
    ph = _t(g.phi).requires_grad_()
    W = _t(case["W"]).requires_grad_()
    m = api.tp_conv(plan, graph, x, ev, ph, W)
    gx, gev, gph, gW = torch.autograd.grad(m, (x, ev, ph, W), _t(case["gout"]), create_graph=True)
    ref = oc.bwd(*oargs(case, prob), case["gout"])
    for name, o in zip(("gx", "gevec", "gphi", "gW"), (gx, gev, gph, gW)):
        assert max_rel(_n(o), ref[name]) <= BWD_TOL, name
    # second order through the edge-vector gradient: d/d(...) of <gev, t>
    t = _t(case["cot"]["evec"])
    h = torch.autograd.grad((gev * t).sum(), (x, ev, ph, W))
    dref = oc.dbwd(*oargs(case, prob), case["gout"], t_gevec=case["cot"]["evec"])
    for name, o in zip(("g_x", "g_evec", "g_phi", "g_W"), h):
        assert max_rel(_n(o), dref[name]) <= BWD_TOL, name


def test_uvu_receiver_route(gpu, monkeypatch):
    """The receiver-state route of channelwise plans (taken when the state-free kernels do not apply),
    forced with SOBEK_UVU_ROUTE=receiver: forward and backward against the oracle."""
    monkeypatch.setenv("SOBEK_UVU_ROUTE", "receiver")
    case = make_case("uvu_small", 120, 1500, 27, isolated=1, mode="uvu")
    api, plan, graph, prob = setup(case)
    g = case["graph"]
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    assert max_rel(_n(api.conv_fwd(plan, graph, *args)), oc.fwd(*oargs(case, prob))) <= FWD_TOL
    ref = oc.bwd(*oargs(case, prob), case["gout"])
    for budget in (0, 1 << 20):
        outs = api.conv_bwd(plan, graph, *args, _t(case["gout"]), budget=budget)
        for name, o in zip(("gx", "gevec", "gphi", "gW"), outs):
            assert max_rel(_n(o), ref[name]) <= BWD_TOL, name
