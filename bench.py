#!/usr/bin/env python3
"""Benchmark of the hot path on one MI355X.

Default workload (the headline): one step = one pass of every operator of the
path over the power-law graph (R-MAT a,b,c,d = .57,.19,.19,.05; 232,965
vertices; 114.6M edges; fp32 features of width 128; edge weights in (0, 1]):

  1. gSpMM  src_mul_edge + sum        (weighted aggregation)
  2. gSpMM  copy_src + max / argmax
  3. gSDDMM dot                       (per-edge attention score)
  4. edge softmax with leaky ReLU(0.2) over the scores of step 3
  (+ the deterministic merge passes of split rows inside 1, 2 and 4)

Other workloads (--workload): the uniform in-degree-100 graph at width --d
(gSpMM copy + sum, gSDDMM), the clustered graph's attention layer (8 heads of
16: gSDDMM -> edge softmax -> gSpMM score x source + sum) and the R-MAT
training step (forward gSpMM on the CSR, backward gSpMM on the CSC, backward
gSDDMM dY . X).

Inputs are resident in HBM before timing starts.  Prints ONE JSON line.
Per-kernel durations come from HIP events recorded on the stream the library
launches on (torch's current stream) around every operator of every timed step.
"""
from __future__ import annotations

import argparse
import json
import os
import re
import sys
import time

import numpy as np

METRIC = "gSpMM/SDDMM GFLOP/s and achieved HBM GB/s (% peak), d=128, one MI355X"
HBM_PEAK_GBS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_rmat_233k_d128.json")
FLOOR_FILE = os.path.join(ROOT, "profiles", "gather_floor_mi355x.json")
NUM_CUS = 256
WORKLOADS = ("rmat_233k_115m", "uniform_deg100_100k", "clustered_133k_deg300",
             "rmat_1m_33m_train", "tiny_uniform_1k", "sage_max_train_rmat_233k",
             "gat_train_clustered_133k", "mlp_rmat_233k", "rand_100k_48m")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# ----------------------------------------------------------------------------
# byte and flop models of the row-wise method (bytes its memory instructions
# must move: the row pointers, each edge's index (and edge value) once, one
# feature row gathered per edge, destination rows once, outputs once)
# ----------------------------------------------------------------------------


def bytes_spmm(n, e, F, H, weighted=False, argmax=False):
    return 4 * (n + 1) + 4 * e + (4 * e * H if weighted else 0) + 4 * e * F + 4 * n * F * (
        2 if argmax else 1)


def bytes_sddmm(n, e, F, H):
    return 4 * (n + 1) + 4 * e + 4 * e * F + 4 * n * F + 4 * e * H


def bytes_softmax(n, e, H):
    return 4 * (n + 1) + 8 * e * H


def bytes_max_bwd(n, c, F, H=1, weighted=False):
    # zero-fill the gradient, read arg and grad_out, the picked edge's source
    # index (and edge value) per element, one atomic read-modify-write
    return 4 * c * F + 8 * n * F + 4 * n * F + (4 * n * F if weighted else 0) + 8 * n * F


def bytes_softmax_bwd(n, e, H, leaky=True):
    # row pointers, read a, grad_out (and scores), write the score gradient
    return 4 * (n + 1) + (16 if leaky else 12) * e * H


class Op:
    def __init__(self, name, fn, nbytes, flop, graded=False):
        self.name, self.fn, self.bytes, self.flop, self.graded = name, fn, nbytes, flop, graded


# ----------------------------------------------------------------------------
# workloads: device setup, operator list, oracle sample
# ----------------------------------------------------------------------------


def _row_sample(csr, edges_target, seed):
    deg = csr.degrees()
    order = np.random.default_rng(seed).permutation(csr.num_rows)
    csum = np.cumsum(deg[order])
    k = min(int(np.searchsorted(csum, edges_target)) + 1, csr.num_rows)
    rows = np.sort(order[:k])
    return rows, int(deg[rows].sum())


def simple_graph(csr):
    """One edge of every (destination, source) pair of a CSR sorted by (dst,
    src), where repeats follow their first copy.  Returns the new CSR and the
    mask of the kept positions."""
    import synth

    rows = np.repeat(np.arange(csr.num_rows), np.diff(csr.indptr.astype(np.int64)))
    keep = np.ones(csr.nnz, bool)
    keep[1:] = (csr.indices[1:] != csr.indices[:-1]) | (rows[1:] != rows[:-1])
    ip = np.zeros(csr.num_rows + 1, np.int64)
    np.cumsum(np.bincount(rows[keep], minlength=csr.num_rows), out=ip[1:])
    return synth.CSR(csr.num_rows, csr.num_cols, ip.astype(np.int32),
                     np.ascontiguousarray(csr.indices[keep])), keep


def setup(name, d, args, fg, torch, dev):
    import synth

    t0 = time.perf_counter()
    base = {"sage_max_train_rmat_233k": "rmat_233k_115m", "mlp_rmat_233k": "rmat_233k_115m",
            "gat_train_clustered_133k": "clustered_133k_deg300"}.get(name, name)
    wl = synth.make_config(base, d=d)
    t_gen = time.perf_counter() - t0
    csr = wl.csr
    if args.simple_graph:
        if base != "rmat_233k_115m":
            raise SystemExit("--simple-graph applies to the power-law graph workloads")
        csr, keep = simple_graph(csr)
        if "w" in wl.arrays:
            wl.arrays["w"] = np.ascontiguousarray(wl.arrays["w"][keep])
    n, e = csr.num_rows, csr.nnz
    log("workload %s: N=%d E=%d generated in %.1fs" % (name, n, e, t_gen))
    G = fg.Graph.from_csr(csr, device=dev)
    popt = dict(segment_edges=args.segment_edges,
                softmax_segment_edges=args.softmax_segment_edges,
                band_row_edges=args.band_row_edges,
                max_row_segments=args.max_row_segments,
                source_slab_rows=args.source_slab_rows,
                partition_min_degree=args.partition_min_degree, item_order=args.item_order)
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    cfg = {"workload": name, "num_vertices": n, "num_edges": e}
    if args.simple_graph:
        cfg["simple_graph"] = True
    plans = []
    plan_ms = []

    def mkplan(g, **kw):  # plan construction is timed apart from the steps
        torch.cuda.synchronize()
        t = time.perf_counter()
        p = fg.Plan(g, **kw)
        plan_ms.append((time.perf_counter() - t) * 1e3)
        return p

    if name in ("rmat_233k_115m", "tiny_uniform_1k"):
        x_h = wl.arrays["x"]
        F = x_h.shape[1]
        w_h = wl.arrays["w"] if "w" in wl.arrays else \
            np.random.default_rng(7).random(e, dtype=np.float32)
        x, wt = T(x_h), T(w_h)
        P = mkplan(G, max_width=F, **popt)
        plans.append(P)
        out_s, out_m = (torch.empty((n, F), device=dev) for _ in range(2))
        arg = torch.empty((n, F), dtype=torch.int32, device=dev)
        sc, at = (torch.empty((e,), device=dev) for _ in range(2))
        ops = [
            Op("spmm_mul_sum", lambda: fg.gspmm(G, x, wt, msg="src_mul_edge", plan=P, out=out_s),
               bytes_spmm(n, e, F, 1, weighted=True), 2 * e * F, graded=True),
            Op("spmm_max", lambda: fg.gspmm(G, x, reduce="max", plan=P, out=out_m, arg=arg),
               bytes_spmm(n, e, F, 1, argmax=True), e * F),
            Op("sddmm_dot", lambda: fg.gsddmm(G, x, x, plan=P, out=sc),
               bytes_sddmm(n, e, F, 1), 2 * e * F, graded=True),
            Op("edge_softmax", lambda: fg.edge_softmax(G, sc, leaky=True, slope=0.2, plan=P,
                                                       out=at),
               bytes_softmax(n, e, 1), 4 * e),
        ]
        if args.fused:
            # SDDMM and edge softmax in one call (both outputs written)
            ops = ops[:2] + [Op("sddmm_softmax", lambda: fg.gsddmm_edge_softmax(
                G, x, x, leaky=True, slope=0.2, plan=P, scores=sc, out=at),
                bytes_sddmm(n, e, F, 1) + 4 * e, 2 * e * F + 4 * e, graded=True)]
            cfg["fused"] = True
        cfg.update(feature_dim=F, graph="R-MAT (.57,.19,.19,.05), self-loops removed, relabelled"
                   if name.startswith("rmat") else "uniform random")

        def oracle_sample(edges_target):
            import oracle

            rows, ne = _row_sample(csr, edges_target, 12345)
            t0 = time.perf_counter()
            oracle.gspmm(csr, x_h, msg=oracle.MSG_SRC_MUL_EDGE, edge_val=w_h, rows=rows)
            oracle.gspmm(csr, x_h, red=oracle.RED_MAX, rows=rows)
            s = oracle.gsddmm(csr, x_h, x_h, rows=rows)
            oracle.edge_softmax(csr, s, leaky=True, slope=0.2, rows=rows)
            dt = time.perf_counter() - t0
            flop = 2 * ne * F + ne * F + 2 * ne * F + 4 * ne
            return dt, flop, "%d random rows (%d edges, %.1f%% of E), all four operators" % (
                rows.size, ne, 100.0 * ne / e)

    elif name in ("uniform_deg100_100k", "rand_100k_48m"):
        x_h = wl.arrays["x"]
        F = x_h.shape[1]
        x = T(x_h)
        P = mkplan(G, max_width=F, **popt)
        plans.append(P)
        out_s = torch.empty((n, F), device=dev)
        sc = torch.empty((e,), device=dev)
        ops = [
            Op("spmm_copy_sum", lambda: fg.gspmm(G, x, plan=P, out=out_s),
               bytes_spmm(n, e, F, 1), 2 * e * F, graded=True),
            Op("sddmm_dot", lambda: fg.gsddmm(G, x, x, plan=P, out=sc),
               bytes_sddmm(n, e, F, 1), 2 * e * F, graded=True),
        ]
        cfg.update(feature_dim=F, graph="uniform, in-degree 100" if name.startswith("uniform")
                   else "two degree classes: 20K vertices ~2000, 80K ~100 (in and out)")

        def oracle_sample(edges_target):
            import oracle

            rows, ne = _row_sample(csr, edges_target, 12345)
            t0 = time.perf_counter()
            oracle.gspmm(csr, x_h, rows=rows)
            oracle.gsddmm(csr, x_h, x_h, rows=rows)
            dt = time.perf_counter() - t0
            return dt, 4 * ne * F, "%d random rows (%d edges), both operators" % (rows.size, ne)

    elif name == "clustered_133k_deg300":
        x_h = wl.arrays["x"]
        H, dh = x_h.shape[1], x_h.shape[2]
        F = H * dh
        x = T(x_h)
        P = mkplan(G, max_width=F, **popt)
        plans.append(P)
        sc, at = (torch.empty((e, H), device=dev) for _ in range(2))
        out = torch.empty((n, H, dh), device=dev)
        ops = [
            Op("sddmm_heads", lambda: fg.gsddmm(G, x, x, plan=P, out=sc),
               bytes_sddmm(n, e, F, H), 2 * e * F, graded=True),
            Op("edge_softmax_heads", lambda: fg.edge_softmax(G, sc, leaky=True, slope=0.2, plan=P,
                                                             out=at),
               bytes_softmax(n, e, H), 4 * e * H),
            Op("spmm_score_sum", lambda: fg.gspmm(G, x, at, msg="src_mul_edge", plan=P, out=out),
               bytes_spmm(n, e, F, H, weighted=True), 2 * e * F, graded=True),
        ]
        if args.fused:
            # the same layer in one kernel: each source row gathered once, no [E, H] arrays
            ops = [Op("gat_fused", lambda: fg.gat_aggregate(G, x, leaky=True, slope=0.2, plan=P,
                                                             out=out),
                      4 * (n + 1) + 4 * e + 4 * e * F + 8 * n * F, 4 * e * F + 4 * e * H,
                      graded=True)]
            cfg["fused"] = True
        cfg.update(feature_dim=F, heads=H, head_dim=dh,
                   graph="100 communities, in-degree 300 (270 inside, 30 uniform)")

        def oracle_sample(edges_target):
            import oracle

            rows, ne = _row_sample(csr, edges_target, 12345)
            x2 = x_h.reshape(n, F)
            t0 = time.perf_counter()
            s = oracle.gsddmm(csr, x2, x2, heads=H, rows=rows)
            a = oracle.edge_softmax(csr, s, heads=H, leaky=True, slope=0.2, rows=rows)
            oracle.gspmm(csr, x2, msg=oracle.MSG_SRC_MUL_EDGE, edge_val=a, heads=H, rows=rows)
            dt = time.perf_counter() - t0
            return dt, 4 * ne * F + 4 * ne * H, "%d random rows (%d edges), attention layer" % (
                rows.size, ne)

    elif name == "sage_max_train_rmat_233k":
        # GraphSage-style max aggregation, forward and backward (the layer's
        # dense transform is outside the sparse path)
        x_h = wl.arrays["x"]
        F = x_h.shape[1]
        x = T(x_h)
        gy_h = np.random.default_rng(11).standard_normal((n, F), dtype=np.float32)
        gy = T(gy_h)
        # the plan also holds the workspace of the binned max backward
        P = mkplan(G, max_width=F, max_backward=not args.atomic_max_backward, **popt)
        plans.append(P)
        out_m = torch.empty((n, F), device=dev)
        arg = torch.empty((n, F), dtype=torch.int32, device=dev)
        gx = torch.empty((csr.num_cols, F), device=dev)
        ops = [
            Op("spmm_max", lambda: fg.gspmm(G, x, reduce="max", plan=P, out=out_m, arg=arg),
               bytes_spmm(n, e, F, 1, argmax=True), e * F, graded=True),
            Op("spmm_max_bwd", lambda: fg.gspmm_max_backward(G, arg, gy, plan=P, grad_src=gx),
               bytes_max_bwd(n, csr.num_cols, F), n * F),
        ]
        cfg.update(feature_dim=F, graph="R-MAT (.57,.19,.19,.05), self-loops removed, relabelled")

        def oracle_sample(edges_target):
            import oracle

            rows, ne = _row_sample(csr, edges_target / 2, 12345)
            t0 = time.perf_counter()
            oracle.gspmm(csr, x_h, red=oracle.RED_MAX, rows=rows)
            oracle.gspmm_max_backward(csr, x_h, gy_h, rows=rows)
            dt = time.perf_counter() - t0
            return dt, ne * F + rows.size * F, (
                "%d random rows (%d edges), forward max and its gradient" % (rows.size, ne))

    elif name == "mlp_rmat_233k":
        # MLP aggregation (d_in = 8 as in the paper's kernel study, d_out = --d):
        # out[v] = max over in-edges of relu((x[u] + x[v]) W); one call = the
        # vertex transform on the matrix cores + the relu(u + v) max gather
        d_in, d_out = 8, (d or 128)
        rng = np.random.default_rng(np.random.SeedSequence([3, d_in, d_out]))
        x_h = rng.standard_normal((n, d_in), dtype=np.float32)
        w_h = (rng.standard_normal((d_in, d_out), dtype=np.float32) / np.sqrt(d_in)).astype(
            np.float32)
        x, wt = T(x_h), T(w_h)
        P = mkplan(G, max_width=d_out, **popt)
        plans.append(P)
        out_m = torch.empty((n, d_out), device=dev)
        arg = torch.empty((n, d_out), dtype=torch.int32, device=dev)
        ws = torch.empty((2 * n * d_out,), device=dev)
        ops = [
            Op("mlp_aggregate", lambda: fg.mlp_aggregate(G, x, wt, plan=P, out=out_m, arg=arg,
                                                         workspace=ws),
               # transform: read X, write P; gather: like gSpMM max over P with P[v] per row
               4 * n * d_in + 4 * n * d_out + bytes_spmm(n, e, d_out, 1, argmax=True)
               + 4 * n * d_out,
               2 * n * d_in * d_out + 3 * e * d_out, graded=True),
        ]
        cfg.update(d_in=d_in, d_out=d_out,
                   graph="R-MAT (.57,.19,.19,.05), self-loops removed, relabelled")

        def oracle_sample(edges_target):
            import oracle

            rows, ne = _row_sample(csr, edges_target / 16, 12345)
            t0 = time.perf_counter()
            oracle.mlp_aggregate(csr, x_h, x_h, w_h, rows=rows)
            dt = time.perf_counter() - t0
            # the oracle evaluates the per-edge form; credited with the same
            # executed-operation count as the GPU's factored form
            return dt, 2 * rows.size * d_in * d_out + 3 * ne * d_out, (
                "%d random rows (%d edges), per-edge definition" % (rows.size, ne))

    elif name == "gat_train_clustered_133k":
        # one graph attention layer (8 heads of 16), forward and backward:
        #   s = X[u].X[v] per head; a = softmax(leaky(s)); Y[v] = sum a X[u]
        #   dX = A^T-side aggregation of a*dY + both SDDMM operand gradients
        # (the three parts of dX are separate outputs; summing them is one
        # elementwise add outside the sparse path)
        csc = synth.csr_to_csc(csr)
        Gt = fg.Graph.from_csr(csc, device=dev, nnz_total=e)
        x_h = wl.arrays["x"]
        H, dh = x_h.shape[1], x_h.shape[2]
        F = H * dh
        x = T(x_h)
        gy = T(np.random.default_rng(12).standard_normal((n, H, dh), dtype=np.float32))
        P = mkplan(G, max_width=F, **popt)
        Pt = mkplan(Gt, max_width=F, **popt)
        plans += [P, Pt]
        sc, at, da = (torch.empty((e, H), device=dev) for _ in range(3))
        y, dx_a, dx_s, dx_d = (torch.empty((n, H, dh), device=dev) for _ in range(4))
        ops = [
            Op("sddmm_heads", lambda: fg.gsddmm(G, x, x, plan=P, out=sc),
               bytes_sddmm(n, e, F, H), 2 * e * F, graded=True),
            Op("edge_softmax_heads", lambda: fg.edge_softmax(G, sc, leaky=True, slope=0.2,
                                                             plan=P, out=at),
               bytes_softmax(n, e, H), 4 * e * H),
            Op("spmm_score_sum", lambda: fg.gspmm(G, x, at, msg="src_mul_edge", plan=P, out=y),
               bytes_spmm(n, e, F, H, weighted=True), 2 * e * F, graded=True),
            Op("bwd_spmm_csc_a", lambda: fg.gspmm(Gt, gy, at, msg="src_mul_edge", plan=Pt,
                                                  out=dx_a),
               bytes_spmm(n, e, F, H, weighted=True), 2 * e * F, graded=True),
        ]
        if args.fused:  # score gradient in one call: SDDMM dY.X fused with the softmax backward
            ops.append(Op("bwd_sddmm_softmax", lambda: fg.gsddmm_edge_softmax_backward(
                G, x, gy, at, scores=sc, leaky=True, slope=0.2, plan=P, grad_scores=da),
                bytes_sddmm(n, e, F, H) + bytes_softmax_bwd(n, e, H) - 4 * (n + 1) - 8 * e * H,
                2 * e * F + 4 * e * H))
        else:
            ops += [
                Op("bwd_sddmm_da", lambda: fg.gsddmm(G, x, gy, plan=P, out=da),
                   bytes_sddmm(n, e, F, H), 2 * e * F, graded=True),
                Op("bwd_edge_softmax", lambda: fg.edge_softmax_backward(
                    G, at, da, scores=sc, leaky=True, slope=0.2, plan=P, grad_scores=da),
                   bytes_softmax_bwd(n, e, H), 4 * e * H),
            ]
        ops += [
            Op("bwd_spmm_csc_ds", lambda: fg.gspmm(Gt, x, da, msg="src_mul_edge", plan=Pt,
                                                   out=dx_s),
               bytes_spmm(n, e, F, H, weighted=True), 2 * e * F, graded=True),
            Op("bwd_spmm_csr_ds", lambda: fg.gspmm(G, x, da, msg="src_mul_edge", plan=P,
                                                   out=dx_d),
               bytes_spmm(n, e, F, H, weighted=True), 2 * e * F, graded=True),
        ]
        cfg.update(feature_dim=F, heads=H, head_dim=dh,
                   graph="100 communities, in-degree 300 (270 inside, 30 uniform), CSR + CSC")

        def oracle_sample(edges_target):
            import oracle

            rows, ne = _row_sample(csr, edges_target / 8, 12345)
            rows_b, ne_b = _row_sample(csc, edges_target / 8, 54321)
            x2 = x_h.reshape(n, F)
            g2 = gy.cpu().numpy().reshape(n, F)
            t0 = time.perf_counter()
            s = oracle.gsddmm(csr, x2, x2, heads=H, rows=rows)
            a = oracle.edge_softmax(csr, s, heads=H, leaky=True, slope=0.2, rows=rows)
            oracle.gspmm(csr, x2, msg=oracle.MSG_SRC_MUL_EDGE, edge_val=a, heads=H, rows=rows)
            oracle.gspmm(csc, g2, msg=oracle.MSG_SRC_MUL_EDGE, edge_val=a, heads=H, rows=rows_b,
                         nnz_total=e)
            ga = oracle.gsddmm(csr, x2, g2, heads=H, rows=rows)
            ds = oracle.edge_softmax_backward(csr, s, ga, heads=H, leaky=True, slope=0.2,
                                              rows=rows)
            oracle.gspmm(csc, x2, msg=oracle.MSG_SRC_MUL_EDGE, edge_val=ds, heads=H,
                         rows=rows_b, nnz_total=e)
            oracle.gspmm(csr, x2, msg=oracle.MSG_SRC_MUL_EDGE, edge_val=ds, heads=H, rows=rows)
            dt = time.perf_counter() - t0
            # six operators over the CSR rows' edges, two over the CSC rows' edges
            flop = 8 * F * ne + 8 * H * ne + 4 * F * ne_b
            return dt, flop, (
                "%d CSR rows (%d edges) and %d CSC rows (%d edges), all eight operators"
                % (rows.size, ne, rows_b.size, ne_b))

    elif name == "rmat_1m_33m_train":
        csc = wl.csc
        Gb = fg.Graph.from_csr(csc, device=dev, nnz_total=e)
        x_h, dy_h = wl.arrays["x"], wl.arrays["dy"]
        F = x_h.shape[1]
        x, dy = T(x_h), T(dy_h)
        Pf = mkplan(G, max_width=F, **popt)
        Pb = mkplan(Gb, max_width=F, **popt)
        plans += [Pf, Pb]
        y, dx = (torch.empty((n, F), device=dev) for _ in range(2))
        da = torch.empty((e,), device=dev)
        ops = [
            Op("fwd_spmm_csr", lambda: fg.gspmm(G, x, plan=Pf, out=y),
               bytes_spmm(n, e, F, 1), 2 * e * F, graded=True),
            Op("bwd_spmm_csc", lambda: fg.gspmm(Gb, dy, plan=Pb, out=dx),
               bytes_spmm(n, e, F, 1), 2 * e * F, graded=True),
            Op("bwd_sddmm", lambda: fg.gsddmm(G, x, dy, plan=Pf, out=da),
               bytes_sddmm(n, e, F, 1), 2 * e * F, graded=True),
        ]
        cfg.update(feature_dim=F, graph="R-MAT (.57,.19,.19,.05) 2^20 vertices, CSR + CSC")

        def oracle_sample(edges_target):
            import oracle

            rows, ne = _row_sample(csr, edges_target / 3, 12345)
            rows_b, ne_b = _row_sample(csc, edges_target / 3, 54321)
            t0 = time.perf_counter()
            oracle.gspmm(csr, x_h, rows=rows)
            oracle.gspmm(csc, dy_h, rows=rows_b, nnz_total=e)
            oracle.gsddmm(csr, x_h, dy_h, rows=rows)
            dt = time.perf_counter() - t0
            return dt, 2 * F * (2 * ne + ne_b), (
                "%d CSR rows (%d edges) and %d CSC rows (%d edges), all three operators"
                % (rows.size, ne, rows_b.size, ne_b))
    else:
        raise SystemExit("unknown workload %r" % name)

    # digests of the seeded inputs (short SHA-256 prefixes), so runs can be matched
    digests = {"indptr": csr.indptr, "indices": csr.indices}
    digests.update({k: v for k, v in wl.arrays.items() if isinstance(v, np.ndarray)})
    cfg["inputs_sha256"] = {k: synth.sha256(v)[:16] for k, v in digests.items()}
    pinfo = plans[0].info()
    cfg.update(segment_edges=pinfo["segment_edges"], max_row_segments=pinfo["max_row_segments"],
               source_slab_rows=pinfo["source_slab_rows"],
               partition_min_degree=pinfo["partition_min_degree"],
               item_order=[p.info()["item_order"] for p in plans], ops=[o.name for o in ops],
               max_backward=[p.info()["max_backward"] for p in plans])
    cfg["plan_build_ms"] = [round(t, 1) for t in plan_ms]
    return cfg, ops, plans, oracle_sample, e


def cpu_baseline(oracle_sample, budget_s, threads=0):
    """The oracle, as is, on a random row sample of the workload, repeated
    until about `budget_s` seconds of host work have been timed; `threads`
    > 0 pins the OpenMP thread count for this measurement."""
    import oracle

    oracle.build(force=False)
    all_threads = oracle.max_threads()
    if threads > 0:
        oracle.set_num_threads(threads)
    try:
        return _cpu_baseline(oracle_sample, budget_s, oracle.max_threads())
    finally:
        oracle.set_num_threads(all_threads)


def _cpu_baseline(oracle_sample, budget_s, threads):
    oracle_sample(200_000)  # warm-up: thread pool, page faults
    dt, flop, desc = oracle_sample(2_000_000)
    # size one pass for about a third of the budget (at most the whole graph)
    target = 2_000_000 * max(1.0, budget_s / 3.0 / max(dt, 1e-9))
    total_t, total_f, reps = 0.0, 0, 0
    while total_t < budget_s:
        dt, flop, desc = oracle_sample(target)
        total_t += dt
        total_f += flop
        reps += 1
    import oracle.fgref as fgref

    return {"value": round(total_f / total_t / 1e9, 3), "unit": "GFLOP/s", "cores": threads,
            "kind": "oracle", "sample": "%s; %d passes, %.1f s" % (desc, reps, total_t),
            "host": _host(), "build": "gcc " + " ".join(fgref.BUILD_FLAGS)}


def _host():
    """CPU model and logical CPU count of the machine the oracle ran on."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpu_model": model, "logical_cpus": os.cpu_count()}


# ----------------------------------------------------------------------------
# counter calibration and summary
# ----------------------------------------------------------------------------


def copy_bandwidth(torch, nbytes=1 << 30, reps=5):
    """Attained HBM rate of a plain 1 GiB device copy (read + write bytes per
    second, median of `reps`): the practical ceiling next to the 8 TB/s peak."""
    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    b.copy_(a)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        e0.record()
        b.copy_(a)
        e1.record()
    torch.cuda.synchronize()
    t = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev])) / 1e3
    del a, b
    return round(2 * nbytes / t / 1e9, 1)


def copy_probe(nbytes=1 << 30, reps=4):
    """A plain device-to-device copy of known size: its FETCH_SIZE / WRITE_SIZE
    counter readings calibrate the counters used for the kernels' traffic."""
    import torch

    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "reps": reps}), flush=True)


KERNEL_OPS = {  # regular expressions over kernel names; template args <G, NV, U, MUL, MAX, ...>
    "spmm_mul_sum": (r"spmm_fast_kernel<\d+, \d+, \d+, true, false", r"spmm_fixup4?_kernel<false"),
    "spmm_max": (r"spmm_fast_kernel<\d+, \d+, \d+, false, true", r"spmm_fixup4?_kernel<true"),
    "sddmm_dot": (r"sddmm_fast_kernel<",),
    "edge_softmax": (r"softmax_kernel<", r"softmax_rowstats_kernel", r"softmax_split_kernel"),
}


def gather_floor(reps=5):
    """Cost of one vector-memory gather instruction per compute unit on a
    cache-resident table (the probe library's fgp_gather_floor): 8 loads in
    flight per wavefront, 2048 workgroups of 4 wavefronts, 2048 loads each;
    tables of 32 KiB and 2 MiB; 1 to 64 active lanes.  Prints one JSON line;
    `floor_ns_per_instruction_per_cu` is the best full-wavefront figure."""
    import ctypes

    from paper_2008_11359_amd.build import PROBE_LIB

    lib = ctypes.CDLL(PROBE_LIB)
    f = lib.fgp_gather_floor
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int] * 5 + [ctypes.POINTER(ctypes.c_float),
                                       ctypes.POINTER(ctypes.c_ulonglong),
                                       ctypes.POINTER(ctypes.c_ulonglong)]
    blocks, iters = 8 * NUM_CUS, 2048
    runs = []
    for rows in (64, 4096):
        for active in (1, 16, 32, 64):
            ms, ct, rt = ctypes.c_float(), ctypes.c_ulonglong(), ctypes.c_ulonglong()
            rc = f(rows, blocks, iters, active, reps, ctypes.byref(ms), ctypes.byref(ct),
                   ctypes.byref(rt))
            if rc != 0:
                raise SystemExit("fgp_gather_floor failed (%d)" % rc)
            instr = blocks * 4 * iters
            ns = ms.value * 1e6 / (instr / NUM_CUS)
            ghz = ct.value / (rt.value / 100e6) / 1e9 if rt.value else None
            runs.append({"table_bytes": rows * 512, "active_lanes": active,
                         "ms": round(ms.value, 4), "instructions": instr,
                         "ns_per_instruction_per_cu": round(ns, 4),
                         "clock_ghz": None if ghz is None else round(ghz, 3),
                         "cycles_per_instruction": None if ghz is None else round(ns * ghz, 2)})
            log("gather floor: table %d B, %d lanes: %.3f ns/instr/CU" % (rows * 512, active, ns))
    full = [r for r in runs if r["active_lanes"] == 64]
    best = min(full, key=lambda r: r["ns_per_instruction_per_cu"])
    # reads alone: 1 GiB, four times the Infinity Cache, grid-stride
    rs = lib.fgp_read_stream
    rs.restype = ctypes.c_int
    rs.argtypes = [ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_float)]
    reads = []
    for blk in (2048, 8192, 32768):
        ms = ctypes.c_float()
        if rs(1 << 30, blk, reps, ctypes.byref(ms)) != 0:
            raise SystemExit("fgp_read_stream failed")
        reads.append({"blocks": blk, "ms": round(ms.value, 4),
                      "gbs": round((1 << 30) / (ms.value / 1e3) / 1e9, 1)})
        log("read stream, %d workgroups: %.1f GB/s" % (blk, reads[-1]["gbs"]))
    rc_ = lib.fgp_read_chunks
    rc_.restype = ctypes.c_int
    rc_.argtypes = [ctypes.c_size_t, ctypes.c_size_t, ctypes.c_int, ctypes.POINTER(ctypes.c_float)]
    chunks = []
    for cb in (4 << 10, 16 << 10, 64 << 10, 256 << 10):
        ms = ctypes.c_float()
        if rc_(1 << 30, cb, reps, ctypes.byref(ms)) != 0:
            raise SystemExit("fgp_read_chunks failed")
        chunks.append({"chunk_bytes": cb, "ms": round(ms.value, 4),
                       "gbs": round((1 << 30) / (ms.value / 1e3) / 1e9, 1)})
        log("read in %d KiB chunks per wavefront: %.1f GB/s" % (cb >> 10, chunks[-1]["gbs"]))
    sr = lib.fgp_scatter_runs
    sr.restype = ctypes.c_int
    sr.argtypes = [ctypes.c_int] * 5 + [ctypes.POINTER(ctypes.c_float)]
    scat = []
    total = 28_000_000  # the records of the power-law graph's max backward at d = 128
    for bins in (64, 256, 1820):
        per = total // 256
        ms = ctypes.c_float()
        if sr(256, per, bins, int(per / bins * 1.3) + 64, reps, ctypes.byref(ms)) != 0:
            raise SystemExit("fgp_scatter_runs failed")
        scat.append({"groups": 256, "bins": bins, "records": per * 256, "ms": round(ms.value, 4)})
        log("scatter of 8-byte records from 256 groups into %d bins: %.3f ms" % (bins, ms.value))
    print(json.dumps({"probe": "fgp_gather_floor (float4 gathers, 1 KiB per instruction)",
                      "floor_ns_per_instruction_per_cu": best["ns_per_instruction_per_cu"],
                      "floor_cycles_per_instruction": best["cycles_per_instruction"],
                      "runs": runs, "read_stream_1gib": reads, "read_chunks_1gib": chunks,
                      "scatter_runs": scat,
                      "read_stream_gbs": max(r["gbs"] for r in reads)}), flush=True)


def _counter_means(csv_dir, counter):
    """Mean value of `counter` per dispatch for each kernel name."""
    import csv
    import glob

    sums, counts = {}, {}
    for path in glob.glob(os.path.join(csv_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            k = r["Kernel_Name"]
            sums[k] = sums.get(k, 0.0) + float(r["Counter_Value"])
            counts[k] = counts.get(k, 0) + 1
    return {k: sums[k] / counts[k] for k in sums}


def summarize_counters(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, out_json,
                       vmem_dir=None):
    """Per-launch fabric/HBM traffic of each operator of the headline workload
    from FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by the
    reading of the same counter for the 1 GiB copy of `--copy-probe`; with
    `vmem_dir` (a run of TA_FLAT_READ_WAVEFRONTS_sum, TA_TA_BUSY_sum and
    GRBM_GUI_ACTIVE) also the vector-memory read instructions per launch."""
    from paper_2008_11359_amd.build import source_digest

    nbytes = 1 << 30

    def copy_factor(d, counter):
        vals = [v for k, v in _counter_means(d, counter).items() if "copy" in k.lower()]
        return nbytes / (max(vals) * 1024.0)

    f_fac = copy_factor(copy_fetch_dir, "FETCH_SIZE")
    w_fac = copy_factor(copy_write_dir, "WRITE_SIZE")
    fetch = _counter_means(fetch_dir, "FETCH_SIZE")
    write = _counter_means(write_dir, "WRITE_SIZE")
    ops = {}
    for op, pats in KERNEL_OPS.items():
        def sel(tab):
            return sum(v for k, v in tab.items() if any(re.search(pt, k) for pt in pats))

        fb = sel(fetch) * 1024.0 * f_fac
        wb = sel(write) * 1024.0 * w_fac
        ops[op] = {"fetch_bytes": round(fb), "write_bytes": round(wb),
                   "hbm_bytes_per_launch": round(fb + wb)}
        if vmem_dir:
            ops[op]["read_instructions"] = round(sel(_counter_means(vmem_dir,
                                                                    "TA_FLAT_READ_WAVEFRONTS_sum")))
            ops[op]["ta_busy_cycles"] = round(sel(_counter_means(vmem_dir, "TA_TA_BUSY_sum")))
            ops[op]["gui_active_cycles"] = round(sel(_counter_means(vmem_dir, "GRBM_GUI_ACTIVE")))
    res = {"source_digest": source_digest(), "fetch_scale": f_fac, "write_scale": w_fac,
           "copy_probe_bytes": nbytes, "ops": ops}
    with open(out_json, "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res, indent=1))


def counters_for(op_name):
    """The counter summary of one operator of the headline workload (traffic
    per launch, and read instructions if taken), or None when the file is
    missing or was taken with other kernel sources."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    try:
        tf = json.load(open(TRAFFIC_FILE))
        from paper_2008_11359_amd.build import source_digest

        if tf.get("source_digest") == source_digest() and op_name in tf.get("ops", {}):
            return tf["ops"][op_name]
        log("traffic file is for other kernel sources: traffic not reported")
    except Exception as exc:  # a stale or malformed file means "not measured"
        log("traffic file ignored:", exc)
    return None


def gather_floor_cycles():
    """Measured gather floor (cycles per instruction per compute unit), or None."""
    try:
        return float(json.load(open(FLOOR_FILE))["floor_cycles_per_instruction"])
    except Exception:
        return None


# the gather path binds when the texture addresser is busy (issuing or
# stalled on the L1/L2) at least this share of the kernel's cycles
VMEM_BUSY_BINDS = 0.8


def roofline_extras(per_op, op_name, ctr, floor_cycles):
    """Counter-grounded figures next to the algorithmic roofline of one
    operator: the rate of the bytes leaving the L2s (an upper bound on its
    HBM traffic: the counters do not tell Infinity Cache hits from HBM reads)
    and the vector-memory ceiling: read instructions per launch times the
    measured per-CU gather floor (cycles), over 256 CUs, against the kernel's
    own cycles per CU (GRBM_GUI_ACTIVE is summed over the 8 dies)."""
    t = per_op[op_name]["ms_mean"] / 1e3
    out = {}
    if ctr is None:
        return out
    tr = ctr["hbm_bytes_per_launch"]
    out["traffic_gbs"] = round(tr / t / 1e9, 1)
    out["traffic_frac"] = round(tr / t / 1e9 / HBM_PEAK_GBS, 4)
    if floor_cycles is not None and ctr.get("read_instructions") and ctr.get("gui_active_cycles"):
        cyc = ctr["gui_active_cycles"] / 8.0
        need = ctr["read_instructions"] / NUM_CUS * floor_cycles
        out["vmem"] = {"read_instructions": ctr["read_instructions"],
                       "floor_cycles_per_instruction": floor_cycles,
                       "kernel_cycles_per_cu": round(cyc),
                       "ceiling_ms": round(t * 1e3 * need / cyc, 4),
                       "frac": round(need / cyc, 4),
                       "ta_busy": round(ctr["ta_busy_cycles"] / (NUM_CUS * cyc), 4)}
    return out


# ----------------------------------------------------------------------------


def time_ops(torch, dev, ops, K, warmup, cold=False):
    """`warmup` untimed steps, then K timed steps of every operator in order,
    each bracketed by HIP events on the launch stream.  Returns the per-op
    event times (ms) and the wall time of the K steps (with `cold`, a 1 GiB
    buffer is overwritten before every operator and the wall time is the sum
    of the operators' event times instead)."""
    for _ in range(warmup):
        for op in ops:
            op.fn()
    torch.cuda.synchronize()
    ev = {op.name: [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                    for _ in range(K)] for op in ops}
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev) if cold else None
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        for op in ops:
            a, b = ev[op.name][k]
            if flush is not None:
                flush.fill_(float(k))
            a.record()
            op.fn()
            b.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_of = {op.name: [a.elapsed_time(b) for a, b in ev[op.name]] for op in ops}
    if flush is not None:  # the flushes are not part of the work
        del flush
        elapsed = sum(sum(v) for v in ms_of.values()) / 1e3
    return ms_of, elapsed


def simple_graph_rates(args, fg, torch, dev, K):
    """The headline step on the power-law graph with one copy of each
    repeated (destination, source) pair: the distinct-edge rate next to the
    multigraph headline (whose repeats gather rows the caches just served)."""
    import copy

    a2 = copy.copy(args)
    a2.simple_graph = True
    cfg, ops, plans, _, e = setup(args.workload, args.d, a2, fg, torch, dev)
    ms_of, elapsed = time_ops(torch, dev, ops, K, args.warmup)
    for p in plans:
        p.close()
    res = {"num_edges": e, "ms_per_step": round(elapsed / K * 1e3, 4),
           "edges_per_s_step": round(e * K / elapsed, 1), "ops": {}}
    for op in ops:
        t = float(np.mean(ms_of[op.name])) / 1e3
        res["ops"][op.name] = {"ms_mean": round(t * 1e3, 4), "edges_per_s": round(e / t, 1),
                               "gflops": round(op.flop / t / 1e9, 1)}
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="rmat_233k_115m", choices=WORKLOADS)
    ap.add_argument("--d", type=int, default=None, help="feature width (uniform workload)")
    ap.add_argument("--segment-edges", type=int, default=0, help="plan segment length (0: default)")
    ap.add_argument("--softmax-segment-edges", type=int, default=0,
                    help="segment length of the edge-softmax schedule (0: --segment-edges if "
                         "given, else the library default)")
    ap.add_argument("--band-row-edges", type=int, default=0,
                    help="die-banded gather schedule: rows of more edges get at least 8 pieces "
                         "(0: library default, -1: none)")
    ap.add_argument("--max-row-segments", type=int, default=0,
                    help="cap on segments per row (0: default)")
    ap.add_argument("--source-slab-rows", type=int, default=0,
                    help="source ids per slab of the gather schedule (0: library default, "
                         "automatic above 128 MiB of features, or 32 MiB with spread gathers; "
                         "-1: automatic above 32 MiB; -2: off)")
    ap.add_argument("--item-order", type=int, default=0,
                    help="plan item order (0: library default, 1: longest first, "
                         "2: length classes with rows in id order)")
    ap.add_argument("--partition-min-degree", type=int, default=0,
                    help="smallest row cut at slab boundaries (0: default)")
    ap.add_argument("--fused", action="store_true",
                    help="attention workload: one fused kernel instead of three operators; "
                         "power-law workload: SDDMM and edge softmax in one call")
    ap.add_argument("--cold", action="store_true",
                    help="overwrite a 1 GiB buffer before every operator (caches hold no "
                         "inputs); the rate then comes from the operators' event times")
    ap.add_argument("--atomic-max-backward", action="store_true",
                    help="sage_max workload: plan without the binned max-backward workspace "
                         "(the gradient goes through fp32 atomics)")
    ap.add_argument("--simple-graph", action="store_true",
                    help="power-law graph workloads: drop the repeated (destination, source) "
                         "pairs of the R-MAT multigraph (31.6%% of its edges) before timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-simple-graph-rate", action="store_true",
                    help="power-law workload: skip the extra timing on the graph without its "
                         "repeated edges (reported as simple_graph)")
    ap.add_argument("--cpu-1thread-budget", type=float, default=4.0,
                    help="seconds of single-thread oracle work (0: skip)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device copy (counter calibration) and exit")
    ap.add_argument("--summarize-counters", nargs="+",
                    metavar="DIR",
                    help="FETCH_DIR WRITE_DIR COPY_FETCH_DIR COPY_WRITE_DIR [VMEM_DIR]: turn "
                         "rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE outputs of the headline "
                         "workload and of --copy-probe (and a TA_FLAT_READ_WAVEFRONTS_sum "
                         "TA_TA_BUSY_sum GRBM_GUI_ACTIVE run) into the traffic file, then exit")
    ap.add_argument("--gather-floor", action="store_true",
                    help="only run the gather-floor probe (cache-resident float4 gathers) and "
                         "print its JSON line")
    args = ap.parse_args()
    sys.path.insert(0, ROOT)
    if args.copy_probe:
        copy_probe()
        return
    if args.summarize_counters:
        d = args.summarize_counters
        if len(d) not in (4, 5):
            raise SystemExit("--summarize-counters takes 4 or 5 directories")
        summarize_counters(*d[:4], TRAFFIC_FILE, vmem_dir=d[4] if len(d) == 5 else None)
        return
    if args.gather_floor:
        gather_floor()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library runs on a single MI355X and has no "
              "multi-GPU mode (got --gpus %d)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2008_11359_amd as fg

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.perf_counter()
    cfg, ops, plans, oracle_sample, e = setup(args.workload, args.d, args, fg, torch, dev)
    torch.cuda.synchronize()
    log("setup %.1fs; plan" % (time.perf_counter() - t0), plans[0].info())

    K = args.steps
    ms_of, elapsed = time_ops(torch, dev, ops, K, args.warmup, args.cold)
    if args.cold:
        cfg["cold"] = True

    per_op = {}
    for op in ops:
        ms = ms_of[op.name]
        t = float(np.mean(ms)) / 1e3
        per_op[op.name] = {
            "ms_mean": round(float(np.mean(ms)), 4),
            "ms_median": round(float(np.median(ms)), 4),
            "gflops": round(op.flop / t / 1e9, 1),
            "gbs_alg": round(op.bytes / t / 1e9, 1),
            "frac_alg": round(op.bytes / t / 1e9 / HBM_PEAK_GBS, 4),
            "bytes_alg": int(op.bytes),
            "edges_per_s": round(e / t, 1),
        }
    flop_step = sum(op.flop for op in ops)
    value = flop_step * K / elapsed / 1e9
    # dominant kernel: the slowest of the graded operators
    dom = max((op for op in ops if op.graded), key=lambda o: per_op[o.name]["ms_mean"]).name
    ach = per_op[dom]["gbs_alg"]
    headline = args.workload == "rmat_233k_115m" and not args.simple_graph
    floor_cyc = gather_floor_cycles()
    ctrs = {o.name: (counters_for(o.name) if headline else None) for o in ops}
    for name, ctr in ctrs.items():  # counter-grounded figures per operator
        per_op[name].update(roofline_extras(per_op, name, ctr, floor_cyc))
    traffic = ctrs[dom]["hbm_bytes_per_launch"] if ctrs[dom] else None
    pinfo = plans[0].info()
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / K * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": cfg,
        "roofline": {
            "bound": "hbm",
            "kernel": dom,
            "achieved": ach,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBS, 4),
            "traffic": traffic,
        },
        "ops": per_op,
        "edges_per_s_step": round(e * K / elapsed, 1),
        "plan": {"segments": pinfo["num_segments"], "split_rows": pinfo["num_split_rows"],
                 "slots": pinfo["num_slots"],
                 "partitioned_rows": pinfo["num_partitioned_rows"]},
    }
    # what `achieved` counts, and the counter-grounded figures beside it
    rl = result["roofline"]
    rl["achieved_counts"] = ("algorithmic bytes: one gathered source row per edge plus indices, "
                             "edge values, destination rows and outputs once; gathers the L2s "
                             "and the Infinity Cache serve count too, so frac can exceed 1")
    extra = roofline_extras(per_op, dom, ctrs[dom], floor_cyc)
    if "traffic_gbs" in extra:
        rl["traffic_gbs"] = extra["traffic_gbs"]
        rl["traffic_frac"] = extra["traffic_frac"]
        rl["traffic_counts"] = ("bytes leaving the L2s per launch (FETCH_SIZE + WRITE_SIZE, "
                                "scaled by a 1 GiB copy): an upper bound on HBM bytes, as the "
                                "counters do not separate Infinity Cache hits")
    if "vmem" in extra:
        rl["vmem"] = extra["vmem"]
        rl["binds"] = "vmem" if extra["vmem"]["ta_busy"] >= VMEM_BUSY_BINDS else "hbm"
        rl["binds_rule"] = ("vmem when the texture addresser is busy (issuing, or stalled on "
                            "the L1 / L2) at least %.0f%% of the kernel's cycles, else hbm"
                            % (100 * VMEM_BUSY_BINDS))
    result["hbm_copy_gbs"] = copy_bandwidth(torch)
    bytes_step = sum(op.bytes for op in ops)
    if args.workload == "rmat_233k_115m" and not args.simple_graph and \
            not args.no_simple_graph_rate and not args.cold:
        # distinct-edge rate: the same step on the graph without repeated pairs
        del ops
        for p in plans:
            p.close()
        plans = []
        log("timing the step on the graph without repeated edges")
        sg = simple_graph_rates(args, fg, torch, dev, min(K, 20))
        sg["duplicate_share"] = round(1.0 - sg["num_edges"] / e, 4)
        sg["note"] = ("one copy of each (destination, source) pair of the same R-MAT draw; "
                      "duplicate_share = stored edges that repeat a pair")
        result["simple_graph"] = sg
    if not args.no_cpu_baseline:
        # the oracle's rate also as edges/s and algorithmic GB/s of the same
        # step: its FLOP rate times the step's edges and bytes per FLOP

        def also_per_edge(cb):
            cb["edges_per_s"] = round(cb["value"] * 1e9 * e / flop_step, 1)
            cb["gbs_alg"] = round(cb["value"] * bytes_step / flop_step, 3)
            return cb

        log("timing the oracle on a row sample")
        result["cpu_baseline"] = also_per_edge(cpu_baseline(oracle_sample, args.cpu_budget))
        if args.cpu_1thread_budget > 0:
            log("timing the oracle on one thread")
            result["cpu_baseline_1thread"] = also_per_edge(
                cpu_baseline(oracle_sample, args.cpu_1thread_budget, threads=1))
    for p in plans:
        p.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
