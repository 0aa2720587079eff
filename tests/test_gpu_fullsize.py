"""GPU parity at the full sizes of the five benchmark workloads.

Each case builds the workload's own graph and tensors (up to 200,000 nodes and
16.0M edges) and runs the library in the launch configuration the benchmark
times: an 8 GiB workspace budget per pass (several receiver chunks on the stress graph), and
for the double backward an edge-vector-only cotangent (the flag set of the
benchmark's "sum of squared edge-vector gradients" loss).  The float64 oracle
cannot run these graphs whole, so the comparison uses outputs it can compute
from a local subgraph:

* forward m and double-backward g_gout at sampled receivers (oracle on their
  in-edges);
* backward phi_bar, evec_bar and double-backward g_phi, g_evec on those
  in-edges;
* x_bar and g_x at sampled senders (oracle on every edge leaving them);
* the global sums A_bar and g_W, and x_bar and g_x as whole tensors, from a
  second full-size run whose output cotangent m_bar is zero outside the sampled
  receivers.  Every backward and double-backward output except g_gout is
  linear in m_bar, so that run must reproduce the oracle on the sampled
  receivers' in-edges and give exactly zero on every other edge.

Tolerances are the same max-norm relative bounds as the small cases.
"""

import numpy as np
import pytest

from oracle import conv as oc
from paper_2607_18074_amd import workloads as wl
from tests.cases import BWD_TOL, FWD_TOL, edge_subgraph, in_edges, max_rel, std_for

pytestmark = pytest.mark.gpu

BUDGET = 8 << 30   # workspace bytes per pass, as in the benchmark

# (sampled receivers, sampled senders); the tiny graph is compared whole
SAMPLES = {"tiny": (None, None), "small": (60, 40), "medium": (32, 20), "wide": (8, 6), "stress": (48, 32)}


def say(*a):
    print(*a, flush=True)


def _check(name, got, ref, tol):
    err = max_rel(got, ref)
    say(f"  {name}: max rel err {err:.2e}")
    assert err <= tol, name


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["tiny", "small", "medium", "wide", "stress"])
def test_full_size(gpu, name):
    import torch
    from paper_2607_18074_amd import api

    cfg = wl.CONFIGS[name]
    sig = (cfg["irreps_in"], cfg["lmax"], cfg["irreps_out"], cfg["K"])
    g = wl.config_graph(name)
    say(f"{name}: N={g.N} E={g.E}")
    std = std_for(cfg["irreps_in"], cfg["irreps_out"], cfg["lmax"], cfg["K"])
    prob = oc.Problem(*sig)
    x = wl.node_features(g.N, prob.dim_in, cfg["index"])
    W = wl.weights(cfg["K"], std, cfg["index"])
    gout = wl.out_cotangent(g.N, prob.dim_out, cfg["index"])
    rdot = wl.cotangents(g.N, g.E, cfg["K"], prob.dim_in, len(std), cfg["index"], which=("evec",))["evec"]

    nr, ns = SAMPLES[name]
    rng = np.random.default_rng(1000 + cfg["index"])
    R = np.arange(g.N) if nr is None else np.sort(rng.choice(g.N, size=nr, replace=False))
    S = np.arange(g.N) if ns is None else np.sort(rng.choice(g.N, size=ns, replace=False))
    gout_m = np.zeros_like(gout)
    gout_m[R] = gout[R]

    # ---- full-size GPU runs -------------------------------------------------------------------
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    N_ = lambda t: t.cpu().numpy()  # noqa: E731
    plan = api.Plan(*sig)
    graph = api.Graph(T(g.rowptr), T(g.sender))
    args = (T(x), T(g.evec), T(g.phi), T(W))
    td = T(rdot)
    say("  gpu fwd (keeping the receiver state, as the benchmark does)")
    state = api.new_state(plan, graph)
    m = N_(api.conv_fwd(plan, graph, *args, budget=BUDGET, state=state))
    say("  gpu bwd / dbwd, dense m_bar (the adjoint state kept by the backward serves the double backward)")
    adj = api.new_state(plan, graph)
    bd = [N_(o) for o in api.conv_bwd(plan, graph, *args, T(gout), budget=BUDGET, state=state, adj_state=adj)]
    dd = [N_(o) for o in api.conv_dbwd(plan, graph, *args, T(gout), t_gevec=td, budget=BUDGET, adj_state=adj)]
    say("  gpu bwd / dbwd, m_bar restricted to the sampled receivers")
    bm = [N_(o) for o in api.conv_bwd(plan, graph, *args, T(gout_m), budget=BUDGET, state=state, adj_state=adj)]
    bm_recompute = N_(api.conv_bwd(plan, graph, *args, T(gout_m), need=(False, False, False, True),
                                   budget=BUDGET)[3])
    dm = [N_(o) for o in api.conv_dbwd(plan, graph, *args, T(gout_m), t_gevec=td, budget=BUDGET, adj_state=adj)]
    dm_recompute = N_(api.conv_dbwd(plan, graph, *args, T(gout_m), t_gevec=td, budget=BUDGET,
                                    need=(False, True, False, False, False))[1])
    del args, td, graph, state, adj
    torch.cuda.empty_cache()

    # ---- oracle on the sampled receivers' in-edges ---------------------------------------------
    A = in_edges(g, R)
    rp, snd, ev, ph, rec = edge_subgraph(g, A)
    say(f"  oracle on {len(R)} receivers ({len(A)} edges)")
    oa = (prob, x, ev, ph, W, rp, snd)
    m_ref = oc.fwd(*oa)
    b_ref = oc.bwd(*oa, gout[rec])
    d_ref = oc.dbwd(*oa, gout[rec], t_gevec=rdot[A])

    _check("fwd m", m[rec], m_ref, FWD_TOL)
    assert np.all(m[np.setdiff1d(R, rec)] == 0)          # sampled receivers without in-edges
    _check("bwd evec_bar", bd[1][A], b_ref["gevec"], BWD_TOL)
    _check("bwd phi_bar", bd[2][A], b_ref["gphi"], BWD_TOL)
    _check("dbwd g_gout", dd[0][rec], d_ref["g_gout"], BWD_TOL)
    _check("dbwd g_evec", dd[2][A], d_ref["g_evec"], BWD_TOL)
    _check("dbwd g_phi", dd[3][A], d_ref["g_phi"], BWD_TOL)

    # restricted m_bar: whole tensors
    other = np.ones(g.E, bool)
    other[A] = False
    _check("bwd x_bar (restricted m_bar)", bm[0], b_ref["gx"], BWD_TOL)
    _check("bwd A_bar (restricted m_bar, retained S)", bm[3], b_ref["gW"], BWD_TOL)
    _check("bwd A_bar (restricted m_bar, recomputed S)", bm_recompute, b_ref["gW"], BWD_TOL)
    _check("bwd evec_bar (restricted m_bar)", bm[1][A], b_ref["gevec"], BWD_TOL)
    _check("dbwd g_x (restricted m_bar, kept Sbar)", dm[1], d_ref["g_x"], BWD_TOL)
    _check("dbwd g_x (restricted m_bar, recomputed Sbar)", dm_recompute, d_ref["g_x"], BWD_TOL)
    _check("dbwd g_W (restricted m_bar)", dm[4], d_ref["g_W"], BWD_TOL)
    _check("dbwd g_phi (restricted m_bar)", dm[3][A], d_ref["g_phi"], BWD_TOL)
    for nm, t in (("evec_bar", bm[1]), ("phi_bar", bm[2]), ("g_evec", dm[2]), ("g_phi", dm[3])):
        assert np.all(t[other] == 0), nm
    # g_gout does not depend on m_bar
    assert np.array_equal(dm[0], dd[0])

    # ---- oracle on every edge leaving the sampled senders --------------------------------------
    B = np.nonzero(np.isin(g.sender, S))[0]
    rp, snd, ev, ph, rec = edge_subgraph(g, B)
    say(f"  oracle on the out-edges of {len(S)} senders ({len(B)} edges)")
    oa = (prob, x, ev, ph, W, rp, snd)
    b_ref = oc.bwd(*oa, gout[rec])
    d_ref = oc.dbwd(*oa, gout[rec], t_gevec=rdot[B])
    _check("bwd x_bar (sampled senders)", bd[0][S], b_ref["gx"][S], BWD_TOL)
    _check("dbwd g_x (sampled senders)", dd[1][S], d_ref["g_x"][S], BWD_TOL)
