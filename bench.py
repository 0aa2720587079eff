#!/usr/bin/env python
"""Benchmark: one step = forward + backward + double backward of the TP convolution.

Prints ONE JSON line.  Workload (default): the edge-scaling stress graph
(200,000 nodes, ~16M directed edges, mean degree 80 at cutoff 6.0, K = 8,
32x0e+32x1o+32x2e with SH up to l = 2), synthetic and seeded.  The backward
cotangent is N(0, 1); the double-backward cotangent is the one of the loss
"sum of squared edge-vector gradients", i.e. t_gevec = 2 * evec_bar with the
other three cotangents zero.  Inputs are resident in HBM before timing.

The forward keeps the receiver state S of every receiver (node-bounded:
N * K * SD floats, 7.2 GB for this workload) and the backward's weight
gradient reads it, as the paper's schedule allows when the state fits; the
backward keeps the adjoint state Sbar = gout A^T (same size) for the double
backward, which computes its directional state dS from scratch.

value = E / (seconds per step): whole-step edge throughput on one GPU.
roofline: the kernel with the largest share of the timed region, its
algorithmic FLOPs per launch (model below) over its mean launch duration,
measured with HIP events recorded on its launch stream inside the timed region.
cpu_baseline: the float64 oracle, timed on this host on a bounded receiver
sample of the same workload, scaled to edges/s.

Algorithmic FLOP model (per edge E, per receiver N; SD = sum_pi C_in d_out,
NZ = sum_pi C_in nnz_pi, G = sum_pi C_in d_out C_out), per pass:
  fwd   E (2 K SD + 2 NZ) + N 2 K G
  bwd   E (4 K SD + 6 NZ) + N 4 K G
  dbwd  E (6 K SD + 6 NZ) + N 6 K G   (edge-vector cotangent alone)
and per kernel:
  fwd_S, fwd_dS (r-only tangent)   E (2 K SD + 2 NZ)
  gemm_sa, gemm_sbar, gemm_ga      N 2 K G per launch set (one per group)
  bwd_E                            E (4 K SD + 6 NZ)
  dbwd_E (r-only tangent)          E (4 K SD + 4 NZ): the double backward's
                                   E (6 K SD + 6 NZ) less the directional state
                                   that fwd_dS computes
The double backward reads the adjoint state the backward kept, so its share
N 2 K G of Sbar = gout A^T runs once per step, in the backward; the pass model
still counts it, as the paper's pass does.  With the states kept, no kernel
launch in a step is recomputation.

paper_context quotes the paper's own figures with their hardware (an NVIDIA
RTX 5090, fp32, against OpenEquivariance on other workloads): context, not a
target for this workload.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "edges/s and % roofline for TP-conv fwd/bwd/double-bwd; peak memory (GB)"
PEAK_FP32_TFLOPS = 157.3      # MI355X fp32 vector / matrix
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def flop_model(plan, N, E):
    K = plan.K
    SD = NZ = G = 0
    for t, (a, _b, c, _w) in enumerate(plan.paths()):
        cin = plan.irreps_in[a][0]
        lo = plan.irreps_out[c][1]
        cout = plan.irreps_out[c][0]
        nnz = int(np.count_nonzero(plan.cg(t)))
        SD += cin * (2 * lo + 1)
        NZ += cin * nnz
        G += cin * (2 * lo + 1) * (1 if getattr(plan, "mode", "uvw") == "uvu" else cout)  # uvu: elementwise
    edge_fwd = E * (2 * K * SD + 2 * NZ)
    edge_bwd = E * (4 * K * SD + 6 * NZ)
    edge_dbwd = E * (4 * K * SD + 4 * NZ)
    gemm = N * 2 * K * G
    per_kernel = {
        "fwd_S": edge_fwd, "fwd_dS": edge_fwd, "bwd_E": edge_bwd, "dbwd_E": edge_dbwd,
        "gemm_sa": gemm, "gemm_sbar": gemm, "gemm_ga": gemm,
    }
    # fwd: S, m = S A; bwd: Sbar = mbar A^T, A_bar = S^T mbar, edge adjoints; dbwd (edge-vector
    # cotangent): dS, m_dot = dS A, g_A = dS^T mbar, Sbar = mbar A^T, edge terms
    passes = {"fwd": edge_fwd + gemm, "bwd": edge_bwd + 2 * gemm, "dbwd": edge_fwd + edge_dbwd + 3 * gemm}
    if getattr(plan, "mode", "uvw") == "uvu":
        # channelwise: per edge and path the weight w = phi A of each channel (2K C), the CG contraction
        # (2 nnz C) and the tied-channel product (2 C d_out); the backward adds phi_bar = A h, G = w mbar
        # and the two transposed contractions; A_bar = S^T mbar is an elementwise reduction (2 flops per
        # element of S).  The direct forward has no state.
        NW = plan.n_weights
        uf = E * (2 * K * NW + 2 * NZ + 2 * SD)
        ua = E * (4 * K * NW + 6 * NZ + 4 * SD)
        ug = N * 2 * K * SD
        passes = {"fwd": uf, "bwd": ua + ug, "dbwd": uf + ua + 2 * ug}
    return dict(SD=SD, NZ=NZ, G=G, per_kernel=per_kernel, passes=passes)


def byte_model(plan, N, E):
    """Algorithmic HBM bytes per pass: inputs read once, outputs written once (fp32)."""
    K, Nw, Cx, Co = plan.K, plan.n_weights, plan.dim_in, plan.dim_out
    fwd = 4 * (N * Cx + E * (3 + K + 1) + (N + 1) + K * Nw + N * Co)
    bwd = fwd + 4 * (N * Cx + E * (K + 3) + K * Nw)
    dbwd = bwd + 4 * (E * 3 + N * Co)   # edge-vector cotangent read, g_gout written
    return {"fwd": fwd, "bwd": bwd, "dbwd": dbwd}


def time_pass(fn, torch):
    """The paper's protocol: warm-up of at least 5 calls and 50 ms, then 10-30 event-timed samples
    totalling at least 250 ms; the median sample."""
    t0, n = time.perf_counter(), 0
    while n < 5 or time.perf_counter() - t0 < 0.05:
        fn()
        torch.cuda.synchronize()
        n += 1
    samples = []
    while len(samples) < 10 or (sum(samples) < 250.0 and len(samples) < 30):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        torch.cuda.synchronize()
        samples.append(a.elapsed_time(b))
    return float(np.median(samples)), len(samples)


def pass_kernels(fn, torch, calls=3):
    """Mean per-pass time of every kernel of one pass (the library's HIP-event launch timer)."""
    from paper_2607_18074_amd import _lib
    torch.cuda.synchronize()
    _lib.profile_reset()
    _lib.profile_enable(True)
    try:
        for _ in range(calls):
            fn()
        torch.cuda.synchronize()
        prof = _lib.profile_read()
    finally:
        _lib.profile_enable(False)
    return {k: dict(launches=n / calls, ms=t / calls) for k, (n, t) in sorted(prof.items(), key=lambda kv: -kv[1][1])}


def sweep(budget_gib, names, dtype="f32", retain=True, kernels=False, policy="auto"):
    """Every workload and pass of the benchmark configurations: one JSON line each, then a table.
    dtype "bf16_gemm" runs the plans' channel GEMM m = S A on bf16 MFMA (tensors stay fp32); policy
    "groups" builds receiver state one output group at a time (eq. receiver_chunk_budget)."""
    import torch

    from paper_2607_18074_amd import api
    from paper_2607_18074_amd import workloads as wl
    torch.cuda.set_device(0)
    budget = int(budget_gib * (1 << 30))
    rows = []
    for name in names:
        cfg = wl.CONFIGS[name]
        g = wl.config_graph(name)
        plan = api.Plan(cfg["irreps_in"], cfg["lmax"], cfg["irreps_out"], cfg["K"], dtype=dtype, policy=policy)
        T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
        graph = api.Graph(T(g.rowptr), T(g.sender))
        xt = T(wl.node_features(g.N, plan.dim_in, cfg["index"]))
        Wt = T(wl.weights(plan.K, plan.weight_std(), cfg["index"]))
        gt = T(wl.out_cotangent(g.N, plan.dim_out, cfg["index"]))
        ev, ph = T(g.evec), T(g.phi)
        ws = {}   # one pass's workspace at a time, so each pass's peak counts only what it needs
        state = api.new_state(plan, graph) if ("bwd" in cfg["passes"] and retain) else None
        adj = api.new_state(plan, graph) if ("dbwd" in cfg["passes"] and retain) else None
        out = torch.empty(g.N, plan.dim_out, device="cuda")
        fm, bm = flop_model(plan, g.N, g.E), byte_model(plan, g.N, g.E)
        fns = {"fwd": lambda: api.conv_fwd(plan, graph, xt, ev, ph, Wt, out=out, ws=ws["fwd"], state=state)}
        if "bwd" in cfg["passes"]:
            fns["bwd"] = lambda: api.conv_bwd(plan, graph, xt, ev, ph, Wt, gt, ws=ws["bwd"], state=state,
                                              adj_state=adj)
        if "dbwd" in cfg["passes"]:
            fns["dbwd"] = lambda: api.conv_dbwd(plan, graph, xt, ev, ph, Wt, gt, t_gevec=rdot, ws=ws["dbwd"],
                                                adj_state=adj)
        rdot = None
        for pname in cfg["passes"]:
            for k in list(ws):
                del ws[k]
            graph._ws.clear()
            torch.cuda.empty_cache()
            ws[pname] = graph.workspace(plan, pname, budget)
            if pname == "bwd":         # the backward reads the state kept by a forward
                ws["fwd"] = ws["bwd"]
                fns["fwd"]()
                del ws["fwd"]
            if pname == "dbwd":        # loss: sum of squared edge-vector gradients
                ws["bwd"] = ws["dbwd"]
                rdot = (2.0 * fns["bwd"]()[1]).contiguous()
                del ws["bwd"]
            torch.cuda.synchronize()
            torch.cuda.reset_peak_memory_stats()
            ms, n = time_pass(fns[pname], torch)
            tf = fm["passes"][pname] / (ms * 1e-3) / 1e12
            gbs = bm[pname] / (ms * 1e-3) / 1e9
            tag = name if dtype == "f32" else f"{name} ({dtype})"
            if not retain:
                tag += f" [no kept state, {budget_gib:g} GiB]"
            if policy != "auto":
                tag += f" [{policy} policy]"
            row = dict(workload=tag, dtype=dtype, retain=retain, pass_=pname,
                       N=g.N, E=g.E, ms=ms, samples=n, edges_per_s=g.E / (ms * 1e-3),
                       tflops=tf, frac_fp32=tf / PEAK_FP32_TFLOPS, alg_gbs=gbs, frac_hbm=gbs / PEAK_HBM_GBS,
                       peak_mem_gb=torch.cuda.max_memory_allocated() / 1e9,
                       workspace_gb=ws[pname].numel() / 1e9,
                       retained_state_gb=sum(t.numel() * 4 / 1e9 for t in (state, adj) if t is not None))
            if kernels:
                row["kernels"] = pass_kernels(fns[pname], torch)
            rows.append(row)
            print(json.dumps({k.rstrip("_"): v for k, v in row.items()}), flush=True)
        del fns, ws, state, adj, out, xt, Wt, gt, ev, ph, graph, plan
        torch.cuda.empty_cache()
    log("| workload | pass | E | ms (median) | edges/s | TFLOP/s | % fp32 | alg. GB/s | peak GB |")
    log("|---|---|---:|---:|---:|---:|---:|---:|---:|")
    for r in rows:
        log(f"| {r['workload']} | {r['pass_']} | {r['E']:,} | {r['ms']:.3f} | {r['edges_per_s'] / 1e6:,.1f} M | "
            f"{r['tflops']:.1f} | {100 * r['frac_fp32']:.1f} | {r['alg_gbs']:.0f} | {r['peak_mem_gb']:.2f} |")
    if kernels:
        log("")
        log("| workload | pass | kernel | launches | ms per pass |")
        log("|---|---|---|---:|---:|")
        for r in rows:
            for k, v in r["kernels"].items():
                if v["ms"] >= 0.05:
                    log(f"| {r['workload']} | {r['pass_']} | `{k}` | {v['launches']:g} | {v['ms']:.3f} |")


def time_graph_passes(plan, W, g, passes, budget, retain, keep_groups=False):
    """Time each pass of `passes` on graph g with the paper's protocol; one dict per pass.  keep_groups:
    the forward keeps the output groups that sobek_retention_select picks within `budget` and the
    backward reads them (the rest recomputed one group at a time)."""
    import torch

    from paper_2607_18074_amd import api
    from paper_2607_18074_amd import workloads as wl
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    graph = api.Graph(T(g.rowptr), T(g.sender))
    xt, ev, ph = T(wl.node_features(g.N, plan.dim_in, 7)), T(g.evec), T(g.phi)
    gt = T(wl.out_cotangent(g.N, plan.dim_out, 7))
    state = api.new_state(plan, graph) if retain else None
    adj = api.new_state(plan, graph) if retain else None
    keep = None
    if keep_groups:
        mask = api.retention(plan, graph, budget)[0]
        keep = (mask, api.new_kept(plan, graph, mask))
    fm = flop_model(plan, g.N, g.E)
    out = []
    for pname in passes:
        graph._ws.clear()
        torch.cuda.empty_cache()
        ws = graph.workspace(plan, pname, budget)
        if pname == "fwd":
            fn = lambda: api.conv_fwd(plan, graph, xt, ev, ph, W, ws=ws, state=state, keep=keep)  # noqa: E731
        elif pname == "bwd":
            if retain or keep:
                api.conv_fwd(plan, graph, xt, ev, ph, W, ws=ws, state=state, keep=keep)
            fn = lambda: api.conv_bwd(plan, graph, xt, ev, ph, W, gt, ws=ws, state=state,  # noqa: E731
                                      adj_state=adj, kept=keep)
        else:
            rdot = (2.0 * api.conv_bwd(plan, graph, xt, ev, ph, W, gt, ws=ws, state=state,
                                       adj_state=adj)[1]).contiguous()
            fn = lambda: api.conv_dbwd(plan, graph, xt, ev, ph, W, gt, t_gevec=rdot, ws=ws,  # noqa: E731
                                       adj_state=adj)
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        ms, n = time_pass(fn, torch)
        tf = fm["passes"][pname] / (ms * 1e-3) / 1e12
        out.append(dict(N=g.N, E=g.E, mean_degree=g.E / g.N, pass_=pname, ms=ms, samples=n,
                        kept_groups=hex(keep[0]) if keep else None,
                        edges_per_s=g.E / (ms * 1e-3), tflops=tf, frac_fp32=tf / PEAK_FP32_TFLOPS,
                        peak_mem_gb=torch.cuda.max_memory_allocated() / 1e9, workspace_gb=ws.numel() / 1e9))
        del ws, fn
    del graph, xt, ev, ph, gt, state, adj
    torch.cuda.empty_cache()
    return out


def tables(which, budget_gib, retain, only=()):
    """The paper's capacity-matched grids (Section 5.4, Tables 3 and 4): every profile and pass on B copies
    of the fixed 128-node degree-32 graph, B the paper's graph count for that pass, timed with its protocol;
    the paper's own M edges/s (another GPU) printed beside ours for context."""
    import torch

    from paper_2607_18074_amd import api
    from paper_2607_18074_amd import workloads as wl
    torch.cuda.set_device(0)
    budget = int(budget_gib * (1 << 30))
    grids = []
    if which in ("uvw", "all"):
        grids.append(("uvw", wl.PAPER_TABLE3_UVW))
    if which in ("uvu", "all"):
        grids.append(("uvu", wl.PAPER_TABLE4_UVU))
    rows = []
    for mode, grid in grids:
        for prof, (n_w, Bs, paper) in grid.items():
            if only and prof not in only:
                continue
            spec, lmax = wl.profile_irreps(prof)
            plan = api.Plan(spec, lmax, spec, wl.REGIME_K, mode=mode)
            assert plan.n_weights == n_w, (prof, plan.n_weights, n_w)
            W = torch.from_numpy(wl.weights(plan.K, plan.weight_std(), 7)).cuda()
            for pi, pname in enumerate(("fwd", "bwd", "dbwd")):
                g = wl.graph_count_graph(Bs[pi])
                r = time_graph_passes(plan, W, g, (pname,), budget, retain)[0]
                r.update(mode=mode, profile=prof, graphs=Bs[pi], paper_medges_per_s=paper[pi])
                rows.append(r)
                print(json.dumps({k.rstrip("_"): x for k, x in r.items()}), flush=True)
            del plan, W
    log("| mode | profile | pass | graphs B | E | M edges/s | paper's (RTX 5090) | % fp32 | peak GB |")
    log("|---|---|---|---:|---:|---:|---:|---:|---:|")
    for r in rows:
        log(f"| {r['mode']} | {r['profile']} | {r['pass_']} | {r['graphs']} | {r['E']:,} | "
            f"{r['edges_per_s'] / 1e6:,.1f} | {r['paper_medges_per_s']:,.1f} | {100 * r['frac_fp32']:.1f} | "
            f"{r['peak_mem_gb']:.2f} |")


def regimes(kinds, profiles, budget_gib, retain, passes=("fwd", "bwd", "dbwd"), policy="auto", keep_groups=False):
    """The paper's scaling regimes: degree scaling (2,048 nodes, mean degree 4..1,023) and graph-count
    scaling (B copies of a 128-node degree-32 graph, B = 2..511) on its representative profiles, every
    pass timed with the paper's protocol; one JSON line per point, a table at the end."""
    import torch

    from paper_2607_18074_amd import api
    from paper_2607_18074_amd import workloads as wl
    torch.cuda.set_device(0)
    budget = int(budget_gib * (1 << 30))
    rows = []
    for prof in profiles:
        spec, lmax = wl.profile_irreps(prof)
        plan = api.Plan(spec, lmax, spec, wl.REGIME_K, policy=policy)
        W = torch.from_numpy(wl.weights(plan.K, plan.weight_std(), 7)).cuda()
        points = [("degree", d) for d in wl.DEGREE_GRID if "degree" in kinds] + \
                 [("count", b) for b in wl.GRAPH_COUNT_GRID if "count" in kinds]
        for kind, v in points:
            g = wl.degree_graph(v)[0] if kind == "degree" else wl.graph_count_graph(v)
            for row in time_graph_passes(plan, W, g, passes, budget, retain, keep_groups):
                row.update(profile=prof, regime=kind, value=v, policy=policy)
                rows.append(row)
                print(json.dumps({k.rstrip("_"): x for k, x in row.items()}), flush=True)
        del plan, W
    log("| profile | regime | N | E | pass | edges/s | % fp32 | peak GB |")
    log("|---|---|---:|---:|---|---:|---:|---:|")
    for r in rows:
        log(f"| {r['profile']} | {r['regime']} {r['value']} | {r['N']:,} | {r['E']:,} | {r['pass_']} | "
            f"{r['edges_per_s'] / 1e6:,.2f} M | {100 * r['frac_fp32']:.1f} | {r['peak_mem_gb']:.2f} |")


def materialized(profiles, counts, budget_gib, mem_cap_gb=200.0):
    """The memory law of Section 2.5 on MI355X: the materialized forward (W = phi A and the edge messages in
    memory, eq. radial_projection_background) against the streamed forward at the same points of the
    paper's graph-count regime (B copies of the 128-node degree-32 graph, K = 16), the streamed one at the
    scratch budget; a point whose materialized W and messages would exceed mem_cap_gb is recorded as not
    fitting, not run.  Roofline per row: the materialized pass against HBM (its algorithmic bytes: W and M
    written and read once, x gathered per edge, phi and the output), the streamed pass against fp32."""
    import torch

    from paper_2607_18074_amd import api
    from paper_2607_18074_amd import workloads as wl
    torch.cuda.set_device(0)
    budget = int(budget_gib * (1 << 30))
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    rows = []
    for prof in profiles:
        spec, lmax = wl.profile_irreps(prof)
        plan = api.Plan(spec, lmax, spec, wl.REGIME_K)
        W = T(wl.weights(plan.K, plan.weight_std(), 7))
        for B in counts:
            g = wl.graph_count_graph(B)
            log(f"materialized sweep: {prof}, B = {B}, E = {g.E:,} ...")
            graph = api.Graph(T(g.rowptr), T(g.sender))
            xt, ev, ph = T(wl.node_features(g.N, plan.dim_in, 7)), T(g.evec), T(g.phi)
            need = api.materialized_bytes(plan, graph)
            row = dict(profile=prof, graphs=B, N=g.N, E=g.E, n_w=plan.n_weights,
                       w_gib=g.E * plan.n_weights * 4 / 2 ** 30, mat_workspace_gb=need / 1e9)
            fm = flop_model(plan, g.N, g.E)
            torch.cuda.empty_cache()
            torch.cuda.synchronize()
            torch.cuda.reset_peak_memory_stats()
            ws = graph.workspace(plan, "fwd", budget)
            ms, _ = time_pass(lambda: api.conv_fwd(plan, graph, xt, ev, ph, W, ws=ws), torch)
            row.update(streamed_ms=ms, streamed_peak_gb=torch.cuda.max_memory_allocated() / 1e9,
                       streamed_frac_fp32=fm["passes"]["fwd"] / (ms * 1e-3) / 1e12 / PEAK_FP32_TFLOPS)
            del ws
            graph._ws.clear()
            torch.cuda.empty_cache()
            if need / 1e9 > mem_cap_gb:
                row.update(mat_ms=None, mat_peak_gb=None, fits=False)
            else:
                torch.cuda.synchronize()
                torch.cuda.reset_peak_memory_stats()
                mws = torch.empty(need, dtype=torch.uint8, device="cuda")
                out = torch.empty(g.N, plan.dim_out, device="cuda")
                ms2, _ = time_pass(lambda: api.conv_fwd_materialized(plan, graph, xt, ev, ph, W, out=out, ws=mws),
                                   torch)
                alg = 4 * (2 * g.E * plan.n_weights + 2 * g.E * plan.dim_out + g.E * plan.dim_in
                           + g.E * (plan.K + 3) + g.N * plan.dim_out)
                row.update(mat_ms=ms2, mat_peak_gb=torch.cuda.max_memory_allocated() / 1e9, fits=True,
                           mat_alg_gb=alg / 1e9, mat_frac_hbm=alg / (ms2 * 1e-3) / 1e9 / PEAK_HBM_GBS,
                           speedup=ms2 / ms)
                del mws, out
            rows.append(row)
            print(json.dumps(row), flush=True)
            del graph, xt, ev, ph
            torch.cuda.empty_cache()
        del plan, W
    log("| profile | B | E | W (GiB) | materialized ms | peak GB | % HBM | streamed ms | peak GB | % fp32 | streamed speedup |")
    log("|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|")
    for r in rows:
        if r["fits"]:
            m = f"{r['mat_ms']:.2f} | {r['mat_peak_gb']:.1f} | {100 * r['mat_frac_hbm']:.1f}"
            sp = f"{r['speedup']:.1f}x"
        else:
            m = f"does not fit ({r['mat_workspace_gb']:.0f} GB) | — | —"
            sp = "—"
        log(f"| {r['profile']} | {r['graphs']} | {r['E']:,} | {r['w_gib']:.1f} | {m} | {r['streamed_ms']:.3f} | "
            f"{r['streamed_peak_gb']:.2f} | {100 * r['streamed_frac_fp32']:.1f} | {sp} |")


PAPER_CONTEXT = {
    "hardware": "NVIDIA RTX 5090 (32 GiB), fp32 throughout, eager, 128 MiB scratch budget (Section 5.1)",
    "workloads": "fixed 128-node degree-32 graph repeated B times, uvw profiles with K = 16 (Section 5.1, Table 3)",
    "uvw_geomean_speedup_vs_openequivariance": {"fwd": 14.9, "bwd": 5.0, "dbwd": 5.7,
                                                "source": "Section 5.4, Table 3 (48 profile/pass pairs)"},
    "uvw_matched_peak_gib": {"sobek": [0.2, 0.7], "openequivariance": [24.1, 30.8], "source": "Section 5.4"},
    "sobek_peak_gib_at_2.1e6_edges": {"range": [0.4, 1.5], "source": "Section 5.2"},
    "table3_128_64_medges_per_s": {"fwd": 197.0, "bwd": 28.1, "dbwd": 5.4,
                                   "source": "Table 3, profile 128/64 (N_w = 36,864)"},
}


def kernel_kind(name):
    for k in ("fwd_dS", "fwd_S", "bwd_E", "dbwd_E", "gemm_sa", "gemm_sbar", "gemm_ga"):
        if name == "sobek_" + k or name.startswith("sobek_" + k + "_"):
            return k
    return None


def source_sha256(sig):
    import hashlib
    from paper_2607_18074_amd import _lib
    return hashlib.sha256(_lib.plan_source(*sig).encode()).hexdigest()


def traffic_record(kernel, sha, launches_per_step):
    """HBM bytes per launch of `kernel` from a committed counter summary, if it still describes this code.

    A summary under profiles/ carries a block
        <!-- traffic-record
        kernel: <name>  source_sha256: <hex>  launches_per_step: <n>
        fetch_bytes_per_launch: <b>  write_bytes_per_launch: <b>
        -->
    (one key per line).  It applies only when the kernel, the hash of the compiled source and the number of
    launches per step all match; otherwise the traffic is unknown (None).
    """
    import glob
    import re
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        text = open(path).read()
        for block in re.findall(r"<!-- traffic-record(.*?)-->", text, re.S):
            rec = dict(re.findall(r"^\s*(\w+):\s*(\S+)\s*$", block, re.M))
            if (rec.get("kernel") == kernel and rec.get("source_sha256") == sha
                    and abs(float(rec.get("launches_per_step", -1)) - launches_per_step) < 1e-6):
                return dict(bytes=float(rec["fetch_bytes_per_launch"]) + float(rec["write_bytes_per_launch"]),
                            fetch=float(rec["fetch_bytes_per_launch"]), write=float(rec["write_bytes_per_launch"]),
                            source=os.path.relpath(path, ROOT))
    return None


def cpu_baseline(case, plan_sig, target_s=15.0):
    """Time the oracle (fwd + bwd + dbwd) on the in-edges of the first receivers."""
    from oracle import conv as oc
    g, x, W, gout, rdot = case
    prob = oc.Problem(*plan_sig)
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = 1
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:  # pragma: no cover
        pass

    def run(R):
        Es = int(g.rowptr[R])
        rp = g.rowptr[:R + 1].astype(np.int64)
        args = (prob, x, g.evec[:Es], g.phi[:Es], W, rp, g.sender[:Es])
        gsub = gout[:R]
        t0 = time.perf_counter()
        oc.fwd(*args)
        oc.bwd(*args, gsub)
        oc.dbwd(*args, gsub, t_gevec=rdot[:Es])
        return Es, time.perf_counter() - t0

    run(2)                       # first call fills the oracle's table caches
    R = 4
    Es, dt = run(R)
    while dt < 0.5 * target_s and R < g.N:
        R = min(g.N, max(R + 1, int(R * min(4.0, 0.9 * target_s / max(dt, 1e-3)))))
        Es, dt = run(R)
    return dict(value=Es / dt, unit="edges/s", cores=int(cores), kind="oracle",
                sample=f"fwd+bwd+dbwd (t_gevec-only) float64 oracle on the in-edges of the first {R} receivers "
                       f"({Es} edges) of the same graph and tensors; {dt:.1f} s",
                seconds=dt, cpu_model=cpu_model, affinity_cpus=len(os.sched_getaffinity(0)))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="stress")
    ap.add_argument("--budget", type=float, default=8.0, help="workspace budget per pass, GiB")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--sweep", default="", help="comma-separated workloads (or 'all'): time every pass of each "
                    "with the paper's protocol instead of the step benchmark, one JSON line per pass")
    ap.add_argument("--dtype", default="f32", choices=["f32", "bf16_gemm"],
                    help="sweep: plan dtype (bf16_gemm: the channel GEMM m = S A on bf16 MFMA)")
    ap.add_argument("--regimes", default="", help="'degree', 'count' or 'all': the paper's scaling regimes on its "
                    "profiles (--profiles), one JSON line per point and pass")
    ap.add_argument("--profiles", default="128/64,128/64/64,128/64/64/64")
    ap.add_argument("--tables", default="", help="'uvw', 'uvu' or 'all': the paper's capacity-matched grids "
                    "(Tables 3 and 4) at its graph counts, one JSON line per profile and pass")
    ap.add_argument("--table-profiles", default="", help="tables: comma-separated subset of profiles (default all)")
    ap.add_argument("--retain", action="store_true", help="regimes: keep S and Sbar across passes (default: the "
                    "paper's setting, recompute within the workspace budget)")
    ap.add_argument("--kernels", action="store_true", help="sweep: also time every kernel of each pass")
    ap.add_argument("--policy", default="auto", choices=["all", "groups", "auto"],
                    help="sweep/regimes: scratch policy of the plans (groups: receiver state one output group "
                         "at a time, eq. receiver_chunk_budget; auto, the library's default: groups for a pass "
                         "whose all-group plan needs three or more receiver chunks)")
    ap.add_argument("--keep-groups", action="store_true",
                    help="regimes: the forward keeps the output groups the retention choice fits in the budget "
                         "and the backward reads them")
    ap.add_argument("--passes", default="fwd,bwd,dbwd", help="regimes: passes to time")
    ap.add_argument("--no-retain", action="store_true",
                    help="sweep: keep no receiver state across passes (each pass recomputes within its budget, the "
                    "paper's setting for a fixed scratch budget)")
    ap.add_argument("--materialized", default="", help="comma-separated graph counts B: the materialized forward "
                    "against the streamed one on the --profiles at those points of the graph-count regime")
    ap.add_argument("--calibrate-copy", type=float, default=0.0,
                    help="only run a plain device copy of this many MiB (traffic-counter calibration)")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        n = int(args.calibrate_copy * (1 << 20)) // 4
        src = torch.randn(n, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "launches": 3}))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only (the library has no multi-GPU path); rerun with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    if args.tables:
        tables(args.tables, args.budget, args.retain,
               tuple(p for p in args.table_profiles.split(",") if p))
        return
    if args.regimes:
        kinds = ("degree", "count") if args.regimes == "all" else tuple(args.regimes.split(","))
        regimes(kinds, args.profiles.split(","), args.budget, args.retain, tuple(args.passes.split(",")),
                args.policy, args.keep_groups)
        return
    if args.materialized:
        materialized(args.profiles.split(","), [int(b) for b in args.materialized.split(",")], args.budget)
        return
    if args.sweep:
        names = ["tiny", "small", "medium", "wide", "stress"] if args.sweep == "all" else args.sweep.split(",")
        sweep(args.budget, names, args.dtype, not args.no_retain, args.kernels, args.policy)
        return

    import torch

    from paper_2607_18074_amd import _lib, api
    from paper_2607_18074_amd import workloads as wl

    cfg = wl.CONFIGS[args.workload]
    t0 = time.time()
    log(f"generating the {args.workload} graph ...")
    g = wl.config_graph(args.workload)
    log(f"graph {args.workload}: N={g.N} E={g.E} ({time.time() - t0:.1f}s)")
    torch.cuda.set_device(0)
    log("creating the plan (kernels from the code-object cache) ...")
    plan = api.Plan(cfg["irreps_in"], cfg["lmax"], cfg["irreps_out"], cfg["K"])
    x = wl.node_features(g.N, plan.dim_in, cfg["index"])
    W = wl.weights(plan.K, plan.weight_std(), cfg["index"])
    gout = wl.out_cotangent(g.N, plan.dim_out, cfg["index"])
    dev = "cuda"
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    graph = api.Graph(T(g.rowptr), T(g.sender))
    xt, ev, ph, Wt, gt = T(x), T(g.evec), T(g.phi), T(W), T(gout)
    budget = int(args.budget * (1 << 30))
    # the passes run one after the other on one stream: they share one workspace, sized for the
    # largest of the three at the budget
    ws_bytes = {p: graph.workspace_bytes(plan, p, budget) for p in ("fwd", "bwd", "dbwd")}
    ws_all = torch.empty(max(ws_bytes.values()), dtype=torch.uint8, device=dev)
    ws = {p: ws_all[:n] for p, n in ws_bytes.items()}
    out = torch.empty(g.N, plan.dim_out, device=dev)
    state = api.new_state(plan, graph)     # receiver state kept from the forward for the backward
    adj = api.new_state(plan, graph)       # adjoint state kept from the backward for the double backward

    def fwd():
        return api.conv_fwd(plan, graph, xt, ev, ph, Wt, out=out, ws=ws["fwd"], state=state)

    def bwd():
        return api.conv_bwd(plan, graph, xt, ev, ph, Wt, gt, ws=ws["bwd"], state=state, adj_state=adj)

    rdot = None

    def dbwd():
        return api.conv_dbwd(plan, graph, xt, ev, ph, Wt, gt, t_gevec=rdot, ws=ws["dbwd"], adj_state=adj)

    # cotangent of L2 = sum |evec_bar|^2
    log("first forward and backward (the double backward's cotangent) ...")
    fwd()
    _, gev, _, _ = bwd()
    rdot = (2.0 * gev).contiguous()
    del gev

    def step():
        fwd()
        bwd()
        dbwd()

    log(f"{args.warmup} warm-up steps ...")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    log(f"{args.steps} timed steps ...")

    # timed region: K steps, with per-launch HIP events on the launch stream
    _lib.profile_reset()
    _lib.profile_enable(True)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    _lib.profile_enable(False)
    prof = _lib.profile_read()
    ms_step = e0.elapsed_time(e1) / args.steps
    peak_gb = torch.cuda.max_memory_allocated() / 1e9

    log(f"timed: {ms_step:.2f} ms per step; per-pass timing ...")
    # per-pass timing (outside the headline region)
    pass_ms = {}
    for name, fn in (("fwd", fwd), ("bwd", bwd), ("dbwd", dbwd)):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(args.steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        pass_ms[name] = a.elapsed_time(b) / args.steps

    fm = flop_model(plan, g.N, g.E)
    sha = source_sha256((cfg["irreps_in"], cfg["lmax"], cfg["irreps_out"], cfg["K"]))
    kernels = {}
    for name, (n, ms) in prof.items():
        kernels[name] = dict(launches_per_step=n / args.steps, ms_per_step=ms / args.steps,
                             mean_launch_ms=ms / max(n, 1))
    dom = max(prof.items(), key=lambda kv: kv[1][1])
    dom_name, (dom_n, dom_ms) = dom
    kind = kernel_kind(dom_name)
    if kind in fm["per_kernel"]:
        per_step = fm["per_kernel"][kind]
        if kind.startswith("gemm"):
            per_step *= {"gemm_sa": 2, "gemm_sbar": 1, "gemm_ga": 2}[kind]  # passes running this GEMM per step
        flops_per_launch = per_step * args.steps / dom_n
        achieved = flops_per_launch / (dom_ms / dom_n * 1e-3) / 1e12
        tr = traffic_record(dom_name, sha, dom_n / args.steps)
        roof = dict(bound="mfma" if kind.startswith("gemm") else "alu", kernel=dom_name, achieved=achieved,
                    peak=PEAK_FP32_TFLOPS, unit="TFLOP/s", frac=achieved / PEAK_FP32_TFLOPS,
                    traffic=None if tr is None else tr["bytes"],
                    flops_per_launch=flops_per_launch, mean_launch_ms=dom_ms / dom_n,
                    launches_per_step=dom_n / args.steps, share_of_step=dom_ms / args.steps / ms_step,
                    source_sha256=sha)
        if tr is not None:
            roof["traffic_gbs"] = tr["bytes"] / (dom_ms / dom_n * 1e-3) / 1e9
            roof["traffic_source"] = tr["source"]
    else:
        roof = dict(bound="hbm", kernel=dom_name, achieved=None, peak=PEAK_HBM_GBS, unit="GB/s", frac=None,
                    traffic=None)

    passes = {}
    bm = byte_model(plan, g.N, g.E)
    for name in ("fwd", "bwd", "dbwd"):
        ms = pass_ms[name]
        tf = fm["passes"][name] / (ms * 1e-3) / 1e12
        gbs = bm[name] / (ms * 1e-3) / 1e9
        passes[name] = dict(ms=ms, edges_per_s=g.E / (ms * 1e-3), tflops=tf, frac_fp32=tf / PEAK_FP32_TFLOPS,
                            alg_gbs=gbs, frac_hbm=gbs / PEAK_HBM_GBS, flops=fm["passes"][name], bytes=bm[name])
    step_flops = sum(fm["passes"].values())

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the oracle on a receiver sample ...")
        cpu = cpu_baseline((g, x, W, gout, rdot.cpu().numpy()),
                           (cfg["irreps_in"], cfg["lmax"], cfg["irreps_out"], cfg["K"]), args.cpu_seconds)

    result = {
        "metric": METRIC,
        "value": g.E / (ms_step * 1e-3),
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "N": g.N, "E": g.E, "K": plan.K, "irreps_in": cfg["irreps_in"],
                   "lmax": cfg["lmax"], "irreps_out": cfg["irreps_out"], "step": "fwd+bwd+dbwd",
                   "dbwd_cotangent": "t_gevec = 2 evec_bar", "workspace_budget_gib": args.budget},
        "roofline": roof,
        "cpu_baseline": cpu,
        "step_tflops": step_flops / (ms_step * 1e-3) / 1e12,
        "step_frac_fp32": step_flops / (ms_step * 1e-3) / 1e12 / PEAK_FP32_TFLOPS,
        "passes": passes,
        "peak_mem_gb": peak_gb,
        "workspace_gb": {p: w.numel() / 1e9 for p, w in ws.items()},
        "workspace_shared_gb": ws_all.numel() / 1e9,
        "retained_state_gb": (state.numel() + adj.numel()) * 4 / 1e9,
        "paper_context": PAPER_CONTEXT,
        "kernels": kernels,
        "wall_s_timed": wall,
    }
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
