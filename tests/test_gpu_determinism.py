"""Bitwise run-to-run determinism of every conv_* route (the header's promise: identical inputs, plan,
graph and workspace size give bitwise identical results, Section 4.3's fixed reduction orders, no float
atomics).  Two identical calls per route, every output compared with np.array_equal:

* fully connected double backward, all four cotangents and the edge-vector cotangent alone, with the
  adjoint state recomputed and read from a kept one, at one receiver chunk and at many;
* channelwise backward and edge-vector double backward on the state-free kernels (per-wave weight-gradient
  partial rows and their fixed-order reduction; the per-slice edge partials of the multi-block form), in
  both backward forms, and the receiver route taken by general cotangents;
* the bf16 channel-GEMM plan's forward, backward and double backward;
* the passes that run part of their work on the plan's second stream, on a non-default caller stream
  synchronised alone, against the default stream.
"""

import numpy as np
import pytest

from tests.cases import make_case

pytestmark = pytest.mark.gpu


def _t(a):
    import torch
    return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _n(t):
    return None if t is None else t.detach().cpu().numpy()


def _twice(fn):
    a = [_n(o) for o in fn()]
    b = [_n(o) for o in fn()]
    for i, (u, v) in enumerate(zip(a, b)):
        if u is None:
            assert v is None
            continue
        assert np.array_equal(u, v), f"output {i} differs between two identical calls"
    return a


def _setup(case, **kw):
    from paper_2607_18074_amd import api
    irr_in, lmax, irr_out, K = case["sig"]
    plan = api.Plan(irr_in, lmax, irr_out, K, **kw)
    g = case["graph"]
    graph = api.Graph(_t(g.rowptr), _t(g.sender))
    args = (_t(case["x"]), _t(g.evec), _t(g.phi), _t(case["W"]))
    return api, plan, graph, args


@pytest.mark.parametrize("budget", [0, 1 << 20])
def test_uvw_double_backward_bitwise(gpu, budget):
    case = make_case("small", 300, 4000, 41, isolated=2)
    api, plan, graph, args = _setup(case)
    gout = _t(case["gout"])
    c = {k: _t(v) for k, v in case["cot"].items()}
    _twice(lambda: api.conv_dbwd(plan, graph, *args, gout, c["x"], c["evec"], c["phi"], c["W"], budget=budget))
    _twice(lambda: api.conv_dbwd(plan, graph, *args, gout, None, c["evec"], None, None, budget=budget))
    adj = api.new_state(plan, graph)
    api.conv_bwd(plan, graph, *args, gout, adj_state=adj)
    _twice(lambda: api.conv_dbwd(plan, graph, *args, gout, c["x"], c["evec"], c["phi"], c["W"], adj_state=adj,
                                 budget=budget))
    _twice(lambda: api.conv_dbwd(plan, graph, *args, gout, None, c["evec"], None, None, adj_state=adj,
                                 budget=budget))


@pytest.mark.parametrize("form", ["u", "s"])
@pytest.mark.parametrize("sig", ["uvu_small", "uvu_wide"])
def test_uvu_bitwise(gpu, sig, form, monkeypatch):
    monkeypatch.setenv("SOBEK_UVU_FORM", form)
    case = make_case(sig, 150, 2000, 42, isolated=1, mode="uvu")
    api, plan, graph, args = _setup(case, mode="uvu")
    gout = _t(case["gout"])
    c = {k: _t(v) for k, v in case["cot"].items()}
    _twice(lambda: [api.conv_fwd(plan, graph, *args)])
    _twice(lambda: api.conv_bwd(plan, graph, *args, gout))
    _twice(lambda: api.conv_dbwd(plan, graph, *args, gout, None, c["evec"], None, None))
    _twice(lambda: api.conv_dbwd(plan, graph, *args, gout, c["x"], c["evec"], c["phi"], c["W"]))


def test_bf16_gemm_bitwise(gpu):
    case = make_case("small", 300, 4000, 43, isolated=2)
    api, plan, graph, args = _setup(case, dtype="bf16_gemm")
    gout = _t(case["gout"])
    c = {k: _t(v) for k, v in case["cot"].items()}
    _twice(lambda: [api.conv_fwd(plan, graph, *args)])
    _twice(lambda: api.conv_bwd(plan, graph, *args, gout))
    _twice(lambda: api.conv_dbwd(plan, graph, *args, gout, c["x"], c["evec"], c["phi"], c["W"]))


def test_second_stream_joins_caller_stream(gpu):
    """The backward's weight gradient from a kept state and the double backward's dS GEMMs run on a
    second stream of the plan, joined back into the caller's stream: on a non-default caller stream,
    synchronising that stream alone must leave every output complete, bitwise equal to a run on the
    default stream (kept states, a workspace small enough for several double-backward chunks)."""
    import torch
    case = make_case("small", 300, 4000, 44, isolated=2)
    api, plan, graph, args = _setup(case)
    gout = _t(case["gout"])
    tev = _t(case["cot"]["evec"])

    def run():
        state, adj = api.new_state(plan, graph), api.new_state(plan, graph)
        m = api.conv_fwd(plan, graph, *args, state=state)
        b = api.conv_bwd(plan, graph, *args, gout, state=state, adj_state=adj)
        d = api.conv_dbwd(plan, graph, *args, gout, None, tev, None, None, adj_state=adj, budget=1 << 20)
        return [m, *b, *d]

    ref = [_n(o) for o in run()]
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        outs = run()
    s.synchronize()
    got = [o.cpu().numpy() if o is not None else None for o in outs]   # copies on the current stream
    for i, (a, b) in enumerate(zip(ref, got)):
        if a is None:
            assert b is None
            continue
        assert np.array_equal(a, b), f"output {i} differs on a non-default caller stream"
