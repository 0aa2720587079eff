"""GPU parity on every operator signature the scaling and capacity sweeps time.

The paper's Table 3 (fully connected ``uvw``, 16 profiles, which include the
three representative profiles 128/64, 128/64/64 and 128/64/64/64 of its scaling
regimes, Section 5.1) and Table 4 (channelwise ``uvu``, 9 profiles) use equal
input and output irreps, one per order l with parity (-1)^l, spherical harmonics
up to the same order and K = 16 radial features.  Each signature runs forward,
backward and double backward (the edge-vector cotangent alone, which the sweeps
time, and all four cotangents) on a small random graph through the C ABI,
against the float64 oracle, at the default workspace (one receiver chunk) and at
a workspace small enough to split the receivers into several chunks.

Channelwise plans have two forms of the state-free backward edge kernel (all
input irreps per lane, or one input irrep per slice); the form is chosen at plan
creation from the compiled kernels' register use, so every profile runs with
each form forced (SOBEK_UVU_FORM), and the test checks from the launch profile
that the forced kernel ran.  Profiles with more than 64 channels take the
multi-block path (per-block partial sums added by a finishing kernel).
"""

import numpy as np
import pytest

from oracle import conv as oc
from paper_2607_18074_amd import workloads as wl
from tests.cases import BWD_TOL, FWD_TOL, make_case, max_rel

pytestmark = pytest.mark.gpu

K = wl.REGIME_K
UVW = sorted(wl.PAPER_TABLE3_UVW)
UVU = sorted(wl.PAPER_TABLE4_UVU)


def profile_sig(name):
    spec, lmax = wl.profile_irreps(name)
    return (spec, lmax, spec, K)


def _t(a):
    import torch
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _n(t):
    return None if t is None else t.detach().cpu().numpy()


def _check(outs, ref, names, tol, what):
    for name, o in zip(names, outs):
        r = ref[name]
        if np.abs(r).max() == 0:
            assert np.abs(_n(o)).max() == 0, f"{what} {name}"
            continue
        err = max_rel(_n(o), r)
        print(f"{what} {name}: {err:.2e}")
        assert err <= tol, f"{what} {name}"


def _run_all(plan, graph, case, prob, budgets, what):
    from paper_2607_18074_amd import api
    g = case["graph"]
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    oa = (prob, case["x"], g.evec, g.phi, case["W"], g.rowptr, g.sender)
    gout = _t(case["gout"])
    ref_f = oc.fwd(*oa)
    ref_b = oc.bwd(*oa, case["gout"])
    c = case["cot"]
    ref_de = oc.dbwd(*oa, case["gout"], t_gevec=c["evec"])
    ref_da = oc.dbwd(*oa, case["gout"], t_gx=c["x"], t_gevec=c["evec"], t_gphi=c["phi"], t_gW=c["W"])
    for budget in budgets:
        tag = f"{what} budget {budget}"
        out = api.conv_fwd(plan, graph, *args, budget=budget)
        _check([out], {"m": ref_f}, ["m"], FWD_TOL, tag + " fwd")
        outs = api.conv_bwd(plan, graph, *args, gout, budget=budget)
        _check(outs, ref_b, ("gx", "gevec", "gphi", "gW"), BWD_TOL, tag + " bwd")
        outs = api.conv_dbwd(plan, graph, *args, gout, None, _t(c["evec"]), None, None, budget=budget)
        _check(outs, ref_de, ("g_gout", "g_x", "g_evec", "g_phi", "g_W"), BWD_TOL, tag + " dbwd[evec]")
        outs = api.conv_dbwd(plan, graph, *args, gout, _t(c["x"]), _t(c["evec"]), _t(c["phi"]), _t(c["W"]),
                             budget=budget)
        _check(outs, ref_da, ("g_gout", "g_x", "g_evec", "g_phi", "g_W"), BWD_TOL, tag + " dbwd[all]")


def _graph(case):
    from paper_2607_18074_amd import api
    g = case["graph"]
    return api.Graph(_t(g.rowptr), _t(g.sender))


@pytest.mark.parametrize("name", UVW)
def test_table3_uvw_profile(gpu, name):
    from paper_2607_18074_amd import api
    sig = profile_sig(name)
    seed = 300 + UVW.index(name)
    case = make_case(sig, 40, 420, seed, isolated=2)
    plan = api.Plan(sig[0], sig[1], sig[2], K)
    prob = oc.Problem(sig[0], sig[1], sig[2], K)
    assert plan.n_weights == prob.n_w == wl.PAPER_TABLE3_UVW[name][0]
    graph = _graph(case)
    _run_all(plan, graph, case, prob, (0, _small_budget(plan, graph)), f"uvw {name}")


def _small_budget(plan, graph):
    """Twice the largest per-pass minimum workspace (chunks of one receiver): several receiver chunks
    and edge windows on these graphs, and every pass still fits."""
    return 2 * max(graph.workspace_bytes(plan, p, 1) for p in ("fwd", "bwd", "dbwd"))


@pytest.mark.parametrize("form", ["u", "s"])
@pytest.mark.parametrize("name", UVU)
def test_table4_uvu_profile(gpu, name, form, monkeypatch):
    from paper_2607_18074_amd import _lib, api
    monkeypatch.setenv("SOBEK_UVU_FORM", form)
    sig = profile_sig(name)
    seed = 400 + UVU.index(name)
    case = make_case(sig, 36, 380, seed, isolated=2, mode="uvu")
    plan = api.Plan(sig[0], sig[1], sig[2], K, mode="uvu")
    prob = oc.Problem(sig[0], sig[1], sig[2], K, mode="uvu")
    assert plan.n_weights == prob.n_w == wl.PAPER_TABLE4_UVU[name][0]
    graph = _graph(case)
    _lib.profile_reset()
    _lib.profile_enable(True)
    try:
        _run_all(plan, graph, case, prob, (0, _small_budget(plan, graph)), f"uvu {name} form {form}")
        prof = _lib.profile_read()
    finally:
        _lib.profile_enable(False)
    # the forced form's kernels ran (plain and edge-vector-tangent variants), the other form's did not
    other = "s" if form == "u" else "u"
    assert f"sobek_uvu_bwd_{form}" in prof and f"sobek_uvu_bwd_{form}t" in prof, sorted(prof)
    assert f"sobek_uvu_bwd_{other}" not in prof and f"sobek_uvu_bwd_{other}t" not in prof, sorted(prof)
