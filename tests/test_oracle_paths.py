"""Pins for path enumeration and weight counts against the numbers the paper prints."""

import json
import os

import pytest

from oracle import irreps as ir

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_weight_counts.json")


def profile_irreps(profile):
    muls = [int(m) for m in profile.split("/")]
    return [(m, l, (-1) ** l) for l, m in enumerate(muls)], len(muls) - 1


def n_w_uvw(profile):
    irr, lmax = profile_irreps(profile)
    return ir.num_weights(ir.enumerate_paths(irr, ir.sh_irreps(lmax), irr))


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_table1_weight_counts_and_memory(golden):
    t = golden["table1"]
    for profile, nw, gib in t["rows"]:
        irr, _ = profile_irreps(profile)
        paths = ir.enumerate_paths(irr, ir.sh_irreps(2), irr)
        assert ir.num_weights(paths) == nw, profile
        # fp32 materialised W at 1e6 edges: 4 E N_w bytes
        assert round(4 * t["edges"] * nw / 2 ** 30, 1) == gib


def test_representative_profiles(golden):
    for profile, nw, edges32 in golden["representative"]["rows"]:
        assert n_w_uvw(profile) == nw
        e = 32 * 2 ** 30 / (4 * nw)
        assert float(f"{e:.1e}") == edges32


def test_table3_weight_counts(golden):
    for profile, nw in golden["table3"]["rows"]:
        assert n_w_uvw(profile) == nw, profile


def test_table4_path_counts(golden):
    # uvu owns C_in weights per path, so N_w / C counts the paths of the same enumeration
    for profile, nw in golden["table4_uvu"]["rows"]:
        irr, lmax = profile_irreps(profile)
        paths = ir.enumerate_paths(irr, ir.sh_irreps(lmax), irr)
        assert len(paths) * irr[0][0] == nw, profile


def test_selection_rules_examples():
    # parity: 1o x 1o can reach 0e, 1e, 2e but not 1o; with no 1e output, 1e is skipped
    irr_in = ir.parse_irreps("1x1o")
    out = ir.parse_irreps("1x0e+1x1o+1x1e+1x2e+1x2o")
    paths = ir.enumerate_paths(irr_in, [(1, 1, -1)], out)
    assert [(p["l_out"], out[p["i_out"]][2]) for p in paths] == [(0, 1), (1, 1), (2, 1)]
    # triangle rule: 2 x 3 cannot reach 0
    paths = ir.enumerate_paths([(1, 2, 1)], [(1, 3, -1)], ir.parse_irreps("1x0o+1x1o+1x5o"))
    assert [p["l_out"] for p in paths] == [1, 5]


def test_weight_offsets_are_cumulative():
    irr = ir.parse_irreps("3x0e+2x1o")
    out = ir.parse_irreps("4x0e+5x1o")
    paths = ir.enumerate_paths(irr, ir.sh_irreps(1), out)
    off = 0
    for p in paths:
        assert p["w_off"] == off and p["n_w"] == p["c_in"] * p["c_out"]
        off += p["n_w"]


def test_layout_roundtrip():
    import numpy as np
    irr = ir.parse_irreps("3x0e+2x1o+1x2e")
    x = np.arange(2 * ir.dim(irr), dtype=float).reshape(2, -1)
    for layout in ("ir_mul", "mul_ir"):
        b = ir.flat_to_blocks(x, irr, layout)
        assert np.array_equal(ir.blocks_to_flat(b, irr, layout), x)
    b = ir.flat_to_blocks(x, irr, "ir_mul")
    # ir_mul: element (u, m) of block 1 sits at 3 + m * 2 + u
    assert b[1][0, 1, 2] == x[0, 3 + 2 * 2 + 1]
    b = ir.flat_to_blocks(x, irr, "mul_ir")
    assert b[1][0, 1, 2] == x[0, 3 + 1 * 3 + 2]
