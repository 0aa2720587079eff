"""Seeded parity cases shared by the GPU tests (inputs only; no method arithmetic)."""

from __future__ import annotations

import numpy as np

from paper_2607_18074_amd import workloads as wl

FWD_TOL = 1e-4   # max-norm relative error, fp32 forward
BWD_TOL = 5e-4   # fp32 backward and double backward

# signatures of the benchmark workloads, reused on small random graphs
SIGS = {
    "tiny": ("8x0e+8x1o", 1, "8x0e+8x1o", 8),
    "small": ("32x0e+32x1o+32x2e", 2, "32x0e+32x1o+32x2e", 8),
    "medium": ("64x0e+64x1o+64x1e+64x2e", 3, "64x0e+64x1o+64x1e+64x2e", 16),
    "wide": ("128x0e+128x1o+128x2e+64x3o", 3, "128x0e+128x1o+128x2e+64x3o", 16),
    # odd multiplicities, a dead input irrep (0o reaches nothing) and a dead output irrep (3e)
    "odd": ("3x0e+5x1o+2x2e+1x0o", 1, "4x0e+3x1o+2x2e+1x3e", 4),
    # an output multiplicity above 256: the adjoint-state GEMM takes the tiled kernel
    "widec": ("320x0e+8x1o", 1, "320x0e+8x1o", 4),
    # channelwise (uvu) signatures: equal multiplicities along every path
    "uvu_small": ("16x0e+16x1o+16x2e", 2, "16x0e+16x1o+16x2e", 8),
    "uvu_l3": ("8x0e+8x1o+8x2e+8x3o", 3, "8x0e+8x1o+8x2e+8x3o", 16),
    "uvu_odd": ("3x0e+3x1o+3x1e+3x2e", 1, "3x0e+3x1o+3x1e+3x2e+1x3e", 4),   # 3e: dead output
    "uvu_wide": ("96x0e+96x1o", 1, "96x0e+96x1o", 4),   # two 64-channel blocks, the second half full
    "uvu_dead": ("4x0e+4x1o+2x0o", 1, "4x0e+4x1o", 4),   # 2x0o reaches no output: zero x-gradient
}


def max_rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.abs(b).max()
    return float(np.abs(a - b).max() / den) if den > 0 else float(np.abs(a).max())


def std_for(irr_in, irr_out, lmax, K, mode="uvw"):
    """Per-weight-column std 1/sqrt(K fan_in) from an independent path count (fan_in: terms summed
    into one output channel, C_in per path for uvw and one per path for uvu)."""
    from oracle import irreps as ir
    paths = ir.enumerate_paths(ir.parse_irreps(irr_in), ir.sh_irreps(lmax), ir.parse_irreps(irr_out), mode)
    fan = {}
    for p in paths:
        fan[p["i_out"]] = fan.get(p["i_out"], 0) + (1 if mode == "uvu" else p["c_in"])
    std = np.zeros(ir.num_weights(paths))
    for p in paths:
        std[p["w_off"]:p["w_off"] + p["n_w"]] = 1.0 / np.sqrt(K * fan[p["i_out"]])
    return std


def make_case(sig, N, E, seed, isolated=0, mode="uvw"):
    """Random receiver-sorted graph (last `isolated` nodes receive nothing) plus all tensors."""
    irr_in, lmax, irr_out, K = SIGS[sig] if isinstance(sig, str) else sig
    from oracle import irreps as ir
    din = ir.dim(ir.parse_irreps(irr_in))
    dout = ir.dim(ir.parse_irreps(irr_out))
    g = wl.random_graph(N, E, seed, K=K, r_c=5.0)
    if isolated:
        # move edges of the last `isolated` receivers onto receiver 0 (keeps the CSR valid)
        recv = np.repeat(np.arange(N), np.diff(g.rowptr))
        recv = np.where(recv >= N - isolated, 0, recv)
        order = np.lexsort((np.arange(len(recv)), g.sender, recv))
        recv, send, ev, ph = recv[order], g.sender[order], g.evec[order], g.phi[order]
        rowptr = np.concatenate([[0], np.cumsum(np.bincount(recv, minlength=N))]).astype(np.int32)
        g = wl.Graph(N, rowptr, send.astype(np.int32), ev, ph)
    std = std_for(irr_in, irr_out, lmax, K, mode)
    x = wl.node_features(N, din, seed)
    W = wl.weights(K, std, seed)
    gout = wl.out_cotangent(N, dout, seed)
    cot = wl.cotangents(N, g.E, K, din, len(std), seed)
    return dict(sig=(irr_in, lmax, irr_out, K), graph=g, x=x, W=W, gout=gout, cot=cot, dim_in=din, dim_out=dout,
                mode=mode)


def edge_subgraph(g, edges):
    """CSR of the edges `edges` (ascending ids of a receiver-sorted graph) with their receivers renumbered.

    Returns (rowptr, sender, evec, phi, receivers): senders keep their node ids, so node tensors are
    passed whole; `receivers[r]` is the original id of renumbered receiver r (row r of a receiver-indexed
    result, and the row to gather from receiver-indexed inputs).
    """
    edges = np.asarray(edges, dtype=np.int64)
    recv = np.repeat(np.arange(g.N), np.diff(g.rowptr))[edges]
    receivers, local = np.unique(recv, return_inverse=True)
    rowptr = np.concatenate([[0], np.cumsum(np.bincount(local, minlength=len(receivers)))]).astype(np.int64)
    return rowptr, g.sender[edges], g.evec[edges], g.phi[edges], receivers


def in_edges(g, receivers):
    """Ids of the edges into `receivers`, ascending."""
    receivers = np.sort(np.asarray(receivers, dtype=np.int64))
    return np.concatenate([np.arange(g.rowptr[r], g.rowptr[r + 1]) for r in receivers]).astype(np.int64)
