"""The generated HIP kernels, run on the CPU by the emulation build (tests/emu), against the oracle.

The emulation library is the library's own host code built against a stand-in HIP runtime; the
plan compiler builds each generated kernel for the host and a wave64 SIMT emulator runs it (every
work-item a fiber; MFMA, shuffles, ballots, readlane and wave barriers synchronise the live lanes of
a wave, __syncthreads the block).  Device buffers sit against inaccessible guard zones and fresh
device memory and every block's LDS are filled with 0xff, so these cases also show that every access
of every launch stays inside its buffer and reads nothing unwritten.  The numerics must match the
float64 oracle within the fp32 tolerances of the GPU parity tests.  Needs the ROCm clang for the
host build; no GPU.
"""

import os
import subprocess
import sys

import numpy as np
import pytest

from oracle import conv as oc
from tests.cases import BWD_TOL, FWD_TOL, make_case, max_rel
from tests.emu import build as emu_build

pytestmark = pytest.mark.skipif(not emu_build.available(), reason="ROCm clang++ not found")


def _run(case, mode="uvw", budgets=(0,)):
    from tests.emu import harness as H
    irr_in, lmax, irr_out, K = case["sig"]
    plan = H.Plan(irr_in, lmax, irr_out, K, mode=mode)
    g = case["graph"]
    graph = H.Graph(g.rowptr, g.sender)
    args = [H.dev(case["x"], "x"), H.dev(g.evec, "evec"), H.dev(g.phi, "phi"), H.dev(case["W"], "W")]
    gout = H.dev(case["gout"], "gout")
    c = case["cot"]
    prob = oc.Problem(irr_in, lmax, irr_out, K, mode=mode)
    oa = (prob, case["x"], g.evec, g.phi, case["W"], g.rowptr, g.sender)
    ref_b = oc.bwd(*oa, case["gout"])
    refs = {"all": oc.dbwd(*oa, case["gout"], t_gx=c["x"], t_gevec=c["evec"], t_gphi=c["phi"], t_gW=c["W"]),
            "evec": oc.dbwd(*oa, case["gout"], t_gevec=c["evec"])}
    for budget in budgets:
        assert max_rel(H.conv_fwd(plan, graph, *args, budget=budget).np(), oc.fwd(*oa)) <= FWD_TOL
        for name, o in zip(("gx", "gevec", "gphi", "gW"), H.conv_bwd(plan, graph, *args, gout, budget=budget)):
            assert max_rel(o.np(), ref_b[name]) <= BWD_TOL, (budget, name)
        for which, ref in refs.items():
            t = [c[k] if which == "all" or k == "evec" else None for k in ("x", "evec", "phi", "W")]
            outs = H.conv_dbwd(plan, graph, *args, gout, *[H.dev(v) for v in t], budget=budget)
            for name, o in zip(("g_gout", "g_x", "g_evec", "g_phi", "g_W"), outs):
                if np.abs(ref[name]).max() == 0:
                    assert np.abs(o.np()).max() == 0, (budget, which, name)
                else:
                    assert max_rel(o.np(), ref[name]) <= BWD_TOL, (budget, which, name)


def test_uvw_tiny_on_emulated_kernels():
    # 8 channels: four MFMA lane blocks per 4x4 tile; the minimum workspace (budget 1) makes the
    # backward run one receiver and one edge window at a time
    _run(make_case("tiny", 48, 600, 81, isolated=2), budgets=(0, 1))


def test_uvw_odd_on_emulated_kernels():
    # odd multiplicities (the VALU path of the state kernel), a dead input and a dead output irrep
    _run(make_case("odd", 40, 500, 82, isolated=1))


@pytest.mark.parametrize("form", ["u", "s"])
def test_uvu_on_emulated_kernels(form, monkeypatch):
    # the state-free channelwise kernels in both backward forms
    monkeypatch.setenv("SOBEK_UVU_FORM", form)
    _run(make_case("uvu_small", 40, 500, 83, isolated=1, mode="uvu"), mode="uvu")


@pytest.mark.parametrize("sig,N,E,seed", [("tiny", 48, 600, 85), ("odd", 40, 500, 86)])
def test_materialized_forward_on_emulated_kernels(sig, N, E, seed):
    # W = phi A and the edge messages formed in the workspace: all edges at once, and edge windows
    # of whole receivers at the smallest workspace the call accepts
    from tests.emu import harness as H
    case = make_case(sig, N, E, seed, isolated=2)
    irr_in, lmax, irr_out, K = case["sig"]
    plan = H.Plan(irr_in, lmax, irr_out, K)
    g = case["graph"]
    graph = H.Graph(g.rowptr, g.sender)
    args = [H.dev(case["x"], "x"), H.dev(g.evec, "evec"), H.dev(g.phi, "phi"), H.dev(case["W"], "W")]
    prob = oc.Problem(irr_in, lmax, irr_out, K)
    ref = oc.fwd(prob, case["x"], g.evec, g.phi, case["W"], g.rowptr, g.sender)
    full = H.materialized_bytes(plan, graph)
    assert full >= E * (plan.n_weights + plan.dim_out) * 4
    for budget in (0, 1):
        out = H.conv_fwd_materialized(plan, graph, *args, budget=budget)
        assert max_rel(out.np(), ref) <= FWD_TOL, budget


def test_guard_zones_catch_an_out_of_bounds_write(tmp_path):
    """The check itself: an output buffer one receiver short makes the forward's last write land in
    the guard zone, which the emulated runtime reports (in a child process, which it ends)."""
    code = f"""
import sys
sys.path.insert(0, {os.path.dirname(os.path.dirname(os.path.abspath(__file__)))!r})
import numpy as np
from tests.cases import make_case
from tests.emu import harness as H
case = make_case("tiny", 16, 100, 84)
irr_in, lmax, irr_out, K = case["sig"]
plan = H.Plan(irr_in, lmax, irr_out, K)
g = case["graph"]
graph = H.Graph(g.rowptr, g.sender)
args = [H.dev(case["x"]), H.dev(g.evec), H.dev(g.phi), H.dev(case["W"])]
out = H.Dev((graph.N - 1, plan.dim_out), np.float32, "short out")
H.conv_fwd(plan, graph, *args, out=out)
print("no fault")
"""
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=600)
    assert r.returncode == 86, (r.returncode, r.stdout[-500:], r.stderr[-2000:])
    assert "buffer" in r.stderr and "short out" in r.stderr and "past the end" in r.stderr, r.stderr[-2000:]
