"""CPU checks of the input recipes (no method arithmetic): the scaling-regime generators realize the
node counts, mean degrees and graph counts of the paper's grids, and produce valid receiver-sorted CSR."""

import numpy as np
import pytest

from paper_2607_18074_amd import workloads as wl


def _check_csr(g):
    assert g.rowptr[0] == 0 and g.rowptr[-1] == g.E
    assert np.all(np.diff(g.rowptr) >= 0)
    assert g.sender.min() >= 0 and g.sender.max() < g.N
    recv = np.repeat(np.arange(g.N), np.diff(g.rowptr))
    assert np.all(recv != g.sender)                        # no self-loops
    assert np.all(np.linalg.norm(g.evec, axis=1) > 1e-6)


@pytest.mark.parametrize("degree", [4, 32, 256, 1023])
def test_degree_grid_realizes_mean_degree(degree):
    g, r_c = wl.degree_graph(degree)
    _check_csr(g)
    assert g.N == 2048
    assert abs(g.E / g.N - degree) <= 0.01 * degree + 0.01
    assert np.all(np.linalg.norm(g.evec, axis=1) < r_c)


def test_degree_grid_is_nested():
    """One position set: a larger cutoff keeps every edge of a smaller one."""
    g1, _ = wl.degree_graph(16)
    g2, _ = wl.degree_graph(64)
    e1 = set(zip(np.repeat(np.arange(g1.N), np.diff(g1.rowptr)).tolist(), g1.sender.tolist()))
    e2 = set(zip(np.repeat(np.arange(g2.N), np.diff(g2.rowptr)).tolist(), g2.sender.tolist()))
    assert e1 <= e2


@pytest.mark.parametrize("B", [2, 13, 511])
def test_graph_count_grid(B):
    g = wl.graph_count_graph(B)
    base = wl.graph_count_graph(1)
    _check_csr(g)
    assert g.N == 128 * B and g.E == B * base.E
    assert 28 <= base.E / base.N <= 36                     # mean degree about 32
    recv = np.repeat(np.arange(g.N), np.diff(g.rowptr))
    assert np.all(recv // 128 == g.sender // 128)          # copies never connect


def test_regime_profiles_match_paper_weight_counts():
    """The profiles' radial-weight counts are the paper's (36,864, 73,728, 131,072)."""
    from oracle import irreps as ir
    want = {"128/64": 36864, "128/64/64": 73728, "128/64/64/64": 131072}
    for name, nw in want.items():
        spec, lmax = wl.profile_irreps(name)
        paths = ir.enumerate_paths(ir.parse_irreps(spec), ir.sh_irreps(lmax), ir.parse_irreps(spec))
        assert ir.num_weights(paths) == nw, name
