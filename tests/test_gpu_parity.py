"""GPU path vs the CPU oracle, through the C ABI (via the ctypes binding).

Tolerance (floating-point sums and dots): |y - ref| <= 1e-5 * sqrt(max(n, 1))
* max(|ref|, ||t||_2), with n the reduction length (in-degree for sums and
softmax, d or dh for dots) and ||t||_2 the L2 norm of the n fp64 terms from the
oracle.  Softmax: |y - ref| <= 1e-5 * sqrt(n) * |ref| + 1e-12.  Max/argmax and
integer-valued inputs: bit-exact.
"""
import ctypes
import math

import numpy as np
import pytest
import torch

import oracle as O
import synth
from synth import csr_rows, csr_to_csc, make_config

pytestmark = pytest.mark.gpu

fg = None  # imported lazily so that collection works without the library


def setup_module(module):
    global fg
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    import paper_2008_11359_amd as _fg

    fg = _fg
    if not __import__("os").path.exists(O.lib_path()):
        O.build()


def say(*a):
    print("[gpu]", *a, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_close_sum(y, ref, tnorm, n):
    y = np.asarray(y, np.float64).reshape(ref.shape)
    n = np.broadcast_to(np.maximum(np.asarray(n, np.float64), 1.0), ref.shape) if np.ndim(n) else \
        np.full(ref.shape, max(float(n), 1.0))
    bound = 1e-5 * np.sqrt(n) * np.maximum(np.abs(ref), tnorm)
    err = np.abs(y - ref)
    bad = err > bound
    assert not bad.any(), "max excess %g at %s (y=%r ref=%r bound=%r)" % (
        (err - bound).max(), np.argwhere(bad)[0], y[bad][0], ref[bad][0], bound[bad][0])


def assert_close_softmax(y, ref, n):
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    bound = 1e-5 * np.sqrt(np.maximum(n, 1)) * np.abs(ref) + 1e-12
    bad = np.abs(y - ref) > bound
    assert not bad.any(), "softmax mismatch at %s: %r vs %r" % (np.argwhere(bad)[0], y[bad][0],
                                                                 ref[bad][0])


def row_edges(g, rows):
    """Stored positions of the given rows (in row order)."""
    return np.concatenate([np.arange(g.indptr[r], g.indptr[r + 1]) for r in rows] or
                          [np.zeros(0, np.int64)]).astype(np.int64)


def edge_ids_of(g, pos):
    return pos if g.edge_ids is None else g.edge_ids[pos].astype(np.int64)


def sample_rows(g, k, seed, extra=()):
    rng = np.random.default_rng(seed)
    deg = g.degrees()
    top = np.argsort(-deg, kind="stable")[:8]
    empty = np.nonzero(deg == 0)[0][:4]
    rnd = rng.choice(g.num_rows, size=min(k, g.num_rows), replace=False)
    return np.unique(np.concatenate([top, empty, rnd, np.asarray(extra, np.int64)])).astype(np.int64)


# ----------------------------------------------------------------------------
# one checker per operator, oracle on selected rows
# ----------------------------------------------------------------------------


def check_spmm(csr, G, x, rows=None, plan=None, edge=None, reduce="sum", heads=1,
               nnz_total=None, exact=False):
    F = int(np.prod(x.shape[1:]))
    msg = "copy_src" if edge is None else "src_mul_edge"
    tx = dev(x)
    te = None if edge is None else dev(edge)
    say("gspmm", msg, reduce, "rows=%d nnz=%d F=%d H=%d plan=%s" % (
        csr.num_rows, csr.nnz, F, heads, None if plan is None else plan.info()["segment_edges"]))
    res = fg.gspmm(G, tx, te, msg=msg, reduce=reduce, heads=heads, plan=plan)
    sel = np.arange(csr.num_rows) if rows is None else rows
    kw = dict(msg=O.MSG_COPY_SRC if edge is None else O.MSG_SRC_MUL_EDGE, heads=heads,
              edge_val=None if edge is None else edge.reshape(-1, heads), rows=rows,
              nnz_total=nnz_total)
    x2 = x.reshape(csr.num_cols, F)
    if reduce == "max":
        out, arg = host(res[0]).reshape(csr.num_rows, F), host(res[1]).reshape(csr.num_rows, F)
        ro, ra = O.gspmm(csr, x2, red=O.RED_MAX, **kw)
        np.testing.assert_array_equal(out[sel].view(np.uint32), ro.view(np.uint32))
        np.testing.assert_array_equal(arg[sel], ra)
        return res
    out = host(res).reshape(csr.num_rows, F)
    ro, norm = O.gspmm(csr, x2, red=O.RED_SUM, with_norm=True, **kw)
    if exact:
        np.testing.assert_array_equal(out[sel], ro)
    else:
        deg = csr.degrees()[sel][:, None]
        assert_close_sum(out[sel], ro.astype(np.float64), norm, deg)
    return res


def check_sddmm(csr, G, xs, xd, rows=None, plan=None, heads=1, nnz_total=None, exact=False):
    F = int(np.prod(xs.shape[1:]))
    say("gsddmm rows=%d nnz=%d F=%d H=%d plan=%s" % (
        csr.num_rows, csr.nnz, F, heads, None if plan is None else plan.info()["segment_edges"]))
    res = fg.gsddmm(G, dev(xs), dev(xd), heads=heads, plan=plan)
    nt = csr.nnz if nnz_total is None else nnz_total
    out = host(res).reshape(nt, heads)
    ro, norm = O.gsddmm(csr, xs.reshape(csr.num_cols, F), xd.reshape(csr.num_rows, F),
                        heads=heads, rows=rows, nnz_total=nt, with_norm=True)
    sel = np.arange(csr.num_rows) if rows is None else rows
    e = edge_ids_of(csr, row_edges(csr, sel))
    if exact:
        np.testing.assert_array_equal(out[e], ro[e])
    else:
        assert_close_sum(out[e], ro[e].astype(np.float64), norm[e], F // heads)
    return res


def check_softmax(csr, G, scores, rows=None, plan=None, heads=1, leaky=True, nnz_total=None):
    say("edge_softmax rows=%d nnz=%d H=%d" % (csr.num_rows, csr.nnz, heads))
    ts = dev(scores)
    res = fg.edge_softmax(G, ts, leaky=leaky, slope=0.2, plan=plan)
    nt = csr.nnz if nnz_total is None else nnz_total
    out = host(res).reshape(nt, heads)
    ro = O.edge_softmax(csr, scores.reshape(nt, heads), heads=heads, leaky=leaky, slope=0.2,
                        rows=rows, nnz_total=nt)
    sel = np.arange(csr.num_rows) if rows is None else rows
    pos = row_edges(csr, sel)
    e = edge_ids_of(csr, pos)
    deg = np.repeat(csr.degrees()[sel], csr.degrees()[sel])[:, None]
    assert_close_softmax(out[e], ro[e], deg)
    return res


def check_sddmm_softmax(csr, G, xs, xd, rows=None, plan=None, heads=1, leaky=True,
                        nnz_total=None):
    """Fused SDDMM + edge softmax vs the oracle's gsddmm and edge_softmax of its
    own scores.  Scores: the SDDMM tolerance.  Weights: the softmax tolerance
    plus the first-order effect of the measured score difference,
    2 * a * max over the row of |leaky(s_gpu) - leaky(s_ref)|."""
    F = int(np.prod(xs.shape[1:]))
    nt = csr.nnz if nnz_total is None else nnz_total
    say("gsddmm_edge_softmax rows=%d nnz=%d F=%d H=%d leaky=%s plan=%s" % (
        csr.num_rows, csr.nnz, F, heads, leaky,
        None if plan is None else plan.info()["segment_edges"]))
    sc, at = fg.gsddmm_edge_softmax(G, dev(xs), dev(xd), heads=heads, leaky=leaky, slope=0.2,
                                    plan=plan)
    sc, at = host(sc).reshape(nt, heads), host(at).reshape(nt, heads)
    x2s, x2d = xs.reshape(csr.num_cols, F), xd.reshape(csr.num_rows, F)
    s_ref, norm = O.gsddmm(csr, x2s, x2d, heads=heads, rows=rows, nnz_total=nt, with_norm=True)
    a_ref = O.edge_softmax(csr, s_ref, heads=heads, leaky=leaky, slope=0.2, rows=rows,
                           nnz_total=nt)
    sel = np.arange(csr.num_rows) if rows is None else rows
    pos = row_edges(csr, sel)
    e = edge_ids_of(csr, pos)
    assert_close_sum(sc[e], s_ref[e].astype(np.float64), norm[e], F // heads)

    def lk(t):
        t = t.astype(np.float64)
        return np.where(t > 0, t, np.float64(np.float32(0.2)) * t) if leaky else t

    d = np.abs(lk(sc[e]) - lk(s_ref[e]))
    deg = csr.degrees()[sel]
    starts = np.concatenate([[0], np.cumsum(deg)[:-1]])
    nz = deg > 0
    dmax = np.zeros((sel.size, heads))
    dmax[nz] = np.maximum.reduceat(d, starts[nz], axis=0)
    dm = np.repeat(dmax, deg, axis=0)
    n = np.repeat(deg, deg)[:, None]
    bound = 1e-5 * np.sqrt(np.maximum(n, 1)) * a_ref[e] + 2 * a_ref[e] * dm + 1e-12
    bad = np.abs(at[e].astype(np.float64) - a_ref[e]) > bound
    assert not bad.any(), "fused softmax mismatch at %s: %r vs %r" % (
        np.argwhere(bad)[0], at[e][bad][0], a_ref[e][bad][0])


def check_gat(csr, G, x, rows=None, plan=None, heads=1, leaky=True):
    """Fused attention aggregation vs the oracle's gsddmm -> edge_softmax ->
    gspmm(src_mul_edge, sum) on the selected rows."""
    F = int(np.prod(x.shape[1:]))
    say("gat_aggregate rows=%d nnz=%d F=%d H=%d plan=%s" % (
        csr.num_rows, csr.nnz, F, heads, None if plan is None else plan.info()["segment_edges"]))
    res = fg.gat_aggregate(G, dev(x), heads=heads, leaky=leaky, slope=0.2, plan=plan)
    out = host(res).reshape(csr.num_rows, F)
    x2 = x.reshape(csr.num_cols, F)
    s = O.gsddmm(csr, x2, x2, heads=heads, rows=rows)
    a = O.edge_softmax(csr, s, heads=heads, leaky=leaky, slope=0.2, rows=rows)
    ro, norm = O.gspmm(csr, x2, msg=O.MSG_SRC_MUL_EDGE, edge_val=a, heads=heads, rows=rows,
                       with_norm=True)
    sel = np.arange(csr.num_rows) if rows is None else rows
    deg = csr.degrees()[sel][:, None]
    assert_close_sum(out[sel], ro.astype(np.float64), norm, deg)
    return res


def _sources_of_ids(csr, nnz_total):
    """source vertex of every edge id (-1 for ids not stored)"""
    src = np.full(nnz_total, -1, np.int64)
    src[edge_ids_of(csr, np.arange(csr.nnz))] = csr.indices
    return src


def check_max_backward(csr, G, x, go, plan=None, edge=None, heads=1, nnz_total=None,
                       exact=False, want_edge=False, bwd_plan=None):
    """gspmm(max) forward on the GPU, then its gradient, vs the oracle's
    gradient (which recomputes the argmax itself).  Term counts for the
    tolerance come from the oracle's own forward.  bwd_plan: a different plan
    for the backward call."""
    F = int(np.prod(x.shape[1:]))
    dh = F // heads
    nt = csr.nnz if nnz_total is None else nnz_total
    msg = "copy_src" if edge is None else "src_mul_edge"
    say("gspmm_max_backward", msg, "rows=%d nnz=%d F=%d H=%d edge_grad=%s plan=%s" % (
        csr.num_rows, csr.nnz, F, heads, want_edge,
        None if plan is None else plan.info()["segment_edges"]))
    tx, te = dev(x), (None if edge is None else dev(edge))
    _, arg = fg.gspmm(G, tx, te, msg=msg, reduce="max", heads=heads, plan=plan)
    res = fg.gspmm_max_backward(G, arg, dev(go), x=tx, edge=te, msg=msg, heads=heads,
                                plan=plan if bwd_plan is None else bwd_plan, want_edge=want_edge)
    gs, ge = (res if want_edge else (res, None))
    gs = host(gs).reshape(csr.num_cols, F)
    x2 = x.reshape(csr.num_cols, F)
    go2 = go.reshape(csr.num_rows, F)
    kw = dict(msg=O.MSG_COPY_SRC if edge is None else O.MSG_SRC_MUL_EDGE, heads=heads,
              edge_val=None if edge is None else edge.reshape(-1, heads), nnz_total=nt)
    if want_edge:
        ge = host(ge).reshape(nt, heads)
    if exact:  # integer-valued terms: any order of the atomic adds gives the same sum
        ref = O.gspmm_max_backward(csr, x2, go2, want_edge=want_edge, **kw)
        rs, re_ = ref if want_edge else (ref, None)
        np.testing.assert_array_equal(gs, rs)
        if want_edge:
            np.testing.assert_array_equal(ge, re_)
        return res
    ref = O.gspmm_max_backward(csr, x2, go2, want_edge=want_edge, with_norm=True, **kw)
    _, ra = O.gspmm(csr, x2, red=O.RED_MAX, **kw)
    sel = ra >= 0
    src = _sources_of_ids(csr, nt)
    fcol = np.broadcast_to(np.arange(F), ra.shape)
    cnt_s = np.zeros((csr.num_cols, F))
    np.add.at(cnt_s, (src[ra[sel]], fcol[sel]), 1.0)
    if want_edge:
        rs, re_, ns, ne = ref
        cnt_e = np.zeros((nt, heads))
        np.add.at(cnt_e, (ra[sel], fcol[sel] // dh), 1.0)
        assert_close_sum(ge, re_.astype(np.float64), ne, cnt_e)
    else:
        rs, ns = ref
    assert_close_sum(gs, rs.astype(np.float64), ns, cnt_s)
    return res


def check_softmax_backward(csr, G, scores, go, rows=None, plan=None, heads=1, leaky=True,
                           nnz_total=None, inplace=False):
    """edge_softmax forward on the GPU, then its gradient from the GPU's
    attention weights, vs the oracle's gradient from the scores.
    Tolerance: |y - ref| <= 1e-5 * sqrt(n) * a (|G| + sum a|G|) + 1e-12."""
    nt = csr.nnz if nnz_total is None else nnz_total
    say("edge_softmax_backward rows=%d nnz=%d H=%d leaky=%s inplace=%s" % (
        csr.num_rows, csr.nnz, heads, leaky, inplace))
    ts, tg = dev(scores), dev(go)
    a = fg.edge_softmax(G, ts, leaky=leaky, slope=0.2, plan=plan)
    ds = fg.edge_softmax_backward(G, a, tg, scores=ts, leaky=leaky, slope=0.2, plan=plan,
                                  grad_scores=tg if inplace else None)
    out = host(ds).reshape(nt, heads)
    ref, scale = O.edge_softmax_backward(csr, scores.reshape(nt, heads), go.reshape(nt, heads),
                                         heads=heads, leaky=leaky, slope=0.2, rows=rows,
                                         nnz_total=nt, with_scale=True)
    sel = np.arange(csr.num_rows) if rows is None else rows
    e = edge_ids_of(csr, row_edges(csr, sel))
    n = np.repeat(csr.degrees()[sel], csr.degrees()[sel])[:, None]
    bound = 1e-5 * np.sqrt(np.maximum(n, 1)) * scale[e] + 1e-12
    err = np.abs(out[e].astype(np.float64) - ref[e])
    bad = err > bound
    assert not bad.any(), "softmax gradient mismatch at %s: %r vs %r (bound %r)" % (
        np.argwhere(bad)[0], out[e][bad][0], ref[e][bad][0], bound[bad][0])
    return ds


def check_sddmm_softmax_backward(csr, G, x, dy, scores, plan=None, leaky=True, nnz_total=None,
                                 rows=None):
    """Score gradient of an attention layer in one call (per-head SDDMM of x
    and dy, then the softmax backward) vs the oracle's SDDMM followed by the
    oracle's softmax backward.  x and dy hold small integers, so the dot
    products are exact on both sides and the softmax-gradient tolerance
    applies: |y - ref| <= 1e-5 * sqrt(n) * a (|G| + sum a|G|) + 1e-12."""
    nt = csr.nnz if nnz_total is None else nnz_total
    heads, dh = x.shape[1], x.shape[2]
    say("gsddmm_edge_softmax_backward rows=%d nnz=%d H=%d dh=%d leaky=%s plan=%s" % (
        csr.num_rows, csr.nnz, heads, dh, leaky,
        None if plan is None else plan.info()["segment_edges"]))
    ts = dev(scores.reshape(nt, heads))
    a = fg.edge_softmax(G, ts, leaky=leaky, slope=0.2, plan=plan)
    ds = host(fg.gsddmm_edge_softmax_backward(G, dev(x), dev(dy), a, scores=ts, leaky=leaky,
                                              slope=0.2, plan=plan)).reshape(nt, heads)
    F = heads * dh
    g_ref = O.gsddmm(csr, x.reshape(csr.num_cols, F), dy.reshape(csr.num_rows, F), heads=heads,
                     nnz_total=nt, rows=rows)
    ref, scale = O.edge_softmax_backward(csr, scores.reshape(nt, heads), g_ref, heads=heads,
                                         leaky=leaky, slope=0.2, nnz_total=nt, with_scale=True,
                                         rows=rows)
    sel = np.arange(csr.num_rows) if rows is None else rows
    e = edge_ids_of(csr, row_edges(csr, sel))
    n = np.repeat(csr.degrees()[sel], csr.degrees()[sel])[:, None]
    bound = 1e-5 * np.sqrt(np.maximum(n, 1)) * scale[e] + 1e-12
    err = np.abs(ds[e].astype(np.float64) - ref[e])
    bad = err > bound
    assert not bad.any(), "attention score gradient mismatch at %s: %r vs %r (bound %r)" % (
        np.argwhere(bad)[0], ds[e][bad][0], ref[e][bad][0], bound[bad][0])
    return ds


def check_dense_matmul(n, d_in, d_out, seed, exact=False):
    rng = np.random.default_rng(seed)
    if exact:
        x = rng.integers(-4, 5, (n, d_in)).astype(np.float32)
        w = rng.integers(-4, 5, (d_in, d_out)).astype(np.float32)
    else:
        x = rng.standard_normal((n, d_in)).astype(np.float32)
        w = rng.standard_normal((d_in, d_out)).astype(np.float32)
    say("dense_matmul n=%d d_in=%d d_out=%d exact=%s" % (n, d_in, d_out, exact))
    y = host(fg.dense_matmul(dev(x), dev(w)))
    ref = O.dense_matmul(x, w)
    if exact:
        np.testing.assert_array_equal(y, ref)
    else:
        tnorm = np.sqrt((x.astype(np.float64) ** 2) @ (w.astype(np.float64) ** 2))
        assert_close_sum(y, ref, tnorm, d_in)


def check_mlp_edges(csr, sel, out, arg):
    """Rules every MLP-aggregation edge must satisfy, whatever the rounding:
    the edge is one of row v's own edges; among duplicate edges (same source,
    so the same message in every rounding) it is the one with the smallest
    id; and where the output is 0 (no positive message, so every message is
    0) it is the row's smallest edge id.  Rows without edges report -1."""
    for i, v in enumerate(sel):
        p0, p1 = int(csr.indptr[v]), int(csr.indptr[v + 1])
        a = arg[i].astype(np.int64)
        if p0 == p1:
            assert (a == -1).all() and (out[i] == 0).all(), "row %d has no edges" % v
            continue
        ids = edge_ids_of(csr, np.arange(p0, p1))
        srcs = csr.indices[p0:p1].astype(np.int64)
        order = np.lexsort((ids, srcs))  # by source, then id
        u_sorted, first = np.unique(srcs[order], return_index=True)
        min_id_of_src = ids[order][first]
        # membership: a's position in this row
        pos_sorted = np.argsort(ids, kind="stable")
        k = np.searchsorted(ids[pos_sorted], a)
        k = np.minimum(k, len(ids) - 1)
        assert (ids[pos_sorted][k] == a).all(), \
            "row %d: edge %r is not an edge of the row" % (v, a[ids[pos_sorted][k] != a][:4])
        src_a = srcs[pos_sorted][k]
        j = np.searchsorted(u_sorted, src_a)
        assert (min_id_of_src[j] == a).all(), \
            "row %d: a duplicate with a smaller id exists for %r" % (v, a[min_id_of_src[j] != a][:4])
        zero = out[i] == 0
        assert (a[zero] == ids.min()).all(), "row %d: zero output must report the smallest id" % v


def check_mlp(csr, G, xs, xd, w, rows=None, plan=None, exact=False, square=False):
    """MLP aggregation vs the oracle's per-edge definition.  Values within the
    rounding of the two forms; the GPU's edge must be an edge of its row,
    attain the oracle's maximum within that tolerance and obey the rules of
    check_mlp_edges; integer inputs: bit-exact values and edges."""
    d_in, d_out = w.shape
    say("mlp_aggregate rows=%d nnz=%d d_in=%d d_out=%d exact=%s plan=%s" % (
        csr.num_rows, csr.nnz, d_in, d_out, exact,
        None if plan is None else plan.info()["segment_edges"]))
    txs = dev(xs)
    out, arg = fg.mlp_aggregate(G, txs, dev(w), x_dst=txs if square else dev(xd), plan=plan)
    out, arg = host(out), host(arg)
    sel = np.arange(csr.num_rows) if rows is None else rows
    ro, ra = O.mlp_aggregate(csr, xs, xd, w, rows=rows)
    out, arg = out[sel], arg[sel]
    if exact:
        np.testing.assert_array_equal(out, ro)
        np.testing.assert_array_equal(arg, ra)
        return
    deg = csr.degrees()[sel]
    assert ((arg >= 0) == (deg > 0)[:, None]).all()
    check_mlp_edges(csr, sel, out, arg)
    # the fp64 message of a given edge id for every (row, feature)
    src = _sources_of_ids(csr, csr.nnz if csr.edge_ids is None else int(csr.edge_ids.max()) + 1)
    w64 = w.astype(np.float64)

    def msg(eids):
        e = np.maximum(eids, 0)
        h = xs[src[e]].astype(np.float64) + xd[sel][:, None, :].astype(np.float64)
        return np.maximum(np.einsum("rik,ki->ri", h, w64), 0.0), \
            np.einsum("rik,ki->ri", np.abs(xs[src[e]].astype(np.float64)) +
                      np.abs(xd[sel][:, None, :].astype(np.float64)), np.abs(w64))

    m_g, _ = msg(arg)
    _, scale = msg(ra)
    tol = 1e-5 * math.sqrt(2 * d_in) * np.maximum(np.abs(ro.astype(np.float64)), scale)
    ne = deg[:, None] > 0
    assert (np.abs(out.astype(np.float64) - ro) <= tol)[ne[:, 0]].all(), "mlp values differ"
    assert (m_g >= ro - tol)[ne[:, 0]].all(), "mlp edge does not attain the maximum"
    np.testing.assert_array_equal(out[~ne[:, 0]], 0)


def plans_for(G, width, sizes=(0, 1, 5, 64)):
    yield None
    for s in sizes:
        yield fg.Plan(G, max_width=width, segment_edges=s)
    # items by length class, rows in id order within a class
    yield fg.Plan(G, max_width=width, segment_edges=64, item_order=2)
    # die-banded pieces of long rows (rows of 8+ pieces at 16-edge pieces)
    yield fg.Plan(G, max_width=width, segment_edges=16, item_order=3)
    # die-banded, every row of more than 20 edges cut into at least 8 pieces
    yield fg.Plan(G, max_width=width, segment_edges=64, item_order=3, band_row_edges=20)
    # rows cut at source-slab boundaries (8 slabs), pieces of at most 64 edges
    slab = max(1, -(-G.num_cols // 8))
    yield fg.Plan(G, max_width=width, segment_edges=64, source_slab_rows=slab,
                  partition_min_degree=1)


# ----------------------------------------------------------------------------
# tiny uniform graph: every operator, exact and rounded inputs, many schedules
# ----------------------------------------------------------------------------


def test_tiny_uniform_all_ops():
    w = make_config("tiny_uniform_1k")
    csr = w.csr
    G = fg.Graph.from_csr(csr)
    x = w.arrays["x"]
    xi = np.random.default_rng(5).integers(-8, 9, size=x.shape).astype(np.float32)
    wgt = np.random.default_rng(6).random(csr.nnz, dtype=np.float32)
    for plan in plans_for(G, 32):
        check_spmm(csr, G, x, plan=plan)
        check_spmm(csr, G, xi, plan=plan, exact=True)
        check_spmm(csr, G, x, plan=plan, reduce="max")
        check_spmm(csr, G, xi, plan=plan, reduce="max")  # many ties
        check_spmm(csr, G, x, plan=plan, edge=wgt)
        check_spmm(csr, G, x, plan=plan, edge=wgt, reduce="max")
        check_sddmm(csr, G, x, x, plan=plan)
        check_sddmm(csr, G, xi, xi, plan=plan, exact=True)
        s_ref = O.gsddmm(csr, x, x)  # the oracle's scores feed both sides
        check_softmax(csr, G, s_ref, plan=plan)
        check_softmax(csr, G, s_ref, plan=plan, leaky=False)


# ----------------------------------------------------------------------------
# widths, heads, fallbacks and edge cases on a small power-law graph
# ----------------------------------------------------------------------------


@pytest.fixture(scope="module")
def small_rmat():
    rng = np.random.default_rng(77)
    csr = synth.rmat_graph(np.random.SeedSequence(77), rng, 11, 2000, 40000)
    deg = csr.degrees()
    assert deg.max() > 500 and (deg == 0).any()
    return csr, fg.Graph.from_csr(csr)


@pytest.mark.parametrize("d", [1, 3, 16, 32, 33, 64, 128, 257, 512, 1040])
def test_widths(small_rmat, d):
    csr, G = small_rmat
    rng = np.random.default_rng(d)
    x = rng.standard_normal((csr.num_cols, d)).astype(np.float32)
    xd = rng.standard_normal((csr.num_rows, d)).astype(np.float32)
    wgt = rng.random(csr.nnz, dtype=np.float32)
    for plan in plans_for(G, d, sizes=(64,)):
        check_spmm(csr, G, x, plan=plan)
        check_spmm(csr, G, x, plan=plan, reduce="max")
        check_spmm(csr, G, x, plan=plan, edge=wgt)
        check_sddmm(csr, G, x, xd, plan=plan)


@pytest.mark.parametrize("heads,dh", [(8, 16), (2, 4), (4, 8), (3, 12), (8, 6), (5, 3), (2, 64),
                                      (70, 2)])
def test_heads(small_rmat, heads, dh):
    csr, G = small_rmat
    rng = np.random.default_rng(heads * 100 + dh)
    x = rng.standard_normal((csr.num_cols, heads, dh)).astype(np.float32)
    x2 = x.reshape(csr.num_cols, heads * dh)
    s_ref = O.gsddmm(csr, x2, x2, heads=heads)  # oracle scores and weights feed both sides
    a_ref = O.edge_softmax(csr, s_ref, heads=heads, leaky=True, slope=0.2)
    for plan in plans_for(G, heads * dh, sizes=(64,)):
        check_sddmm(csr, G, x, x, plan=plan, heads=heads)
        check_softmax(csr, G, s_ref, plan=plan, heads=heads)
        check_spmm(csr, G, x, plan=plan, edge=a_ref, heads=heads)
        check_spmm(csr, G, x, plan=plan, edge=a_ref, heads=heads, reduce="max")


@pytest.mark.parametrize("heads,dh", [(8, 16), (1, 128), (2, 32), (4, 8), (1, 4), (16, 16),
                                      (1, 256), (4, 64), (2, 128), (2, 64), (4, 32), (64, 4)])
def test_gat_fused(small_rmat, heads, dh):
    csr, G = small_rmat
    x = np.random.default_rng(heads * 7 + dh).standard_normal(
        (csr.num_cols, heads, dh)).astype(np.float32)
    for plan in plans_for(G, heads * dh, sizes=(1, 64)):
        check_gat(csr, G, x, plan=plan, heads=heads)
        check_gat(csr, G, x, plan=plan, heads=heads, leaky=False)


@pytest.mark.parametrize("d,heads,weighted", [(1, 1, False), (33, 1, False), (128, 1, False),
                                              (128, 1, True), (48, 8, True), (20, 5, False)])
def test_max_backward(small_rmat, d, heads, weighted):
    csr, G = small_rmat
    rng = np.random.default_rng(d * 10 + heads)
    x = rng.standard_normal((csr.num_cols, d)).astype(np.float32)
    go = rng.standard_normal((csr.num_rows, d)).astype(np.float32)
    xi = rng.integers(-3, 4, (csr.num_cols, d)).astype(np.float32)  # ties
    gi = rng.integers(-8, 9, (csr.num_rows, d)).astype(np.float32)  # exact sums
    w = (rng.random((csr.nnz, heads)) + 0.5).astype(np.float32) if weighted else None
    wi = rng.integers(1, 3, (csr.nnz, heads)).astype(np.float32) if weighted else None
    for plan in (None, fg.Plan(G, max_width=d, segment_edges=64),
                 fg.Plan(G, max_width=d, max_backward=True)):
        check_max_backward(csr, G, x, go, plan=plan, edge=w, heads=heads, want_edge=weighted)
        check_max_backward(csr, G, xi, gi, plan=plan, edge=wi, heads=heads, want_edge=weighted,
                           exact=True)


@pytest.mark.parametrize("heads,leaky", [(1, True), (1, False), (8, True), (3, True), (70, False)])
def test_softmax_backward(small_rmat, heads, leaky):
    csr, G = small_rmat
    rng = np.random.default_rng(heads * 3 + leaky)
    s = (4 * rng.standard_normal((csr.nnz, heads))).astype(np.float32)
    s[rng.random(s.shape) < 0.02] = 0.0
    go = rng.standard_normal((csr.nnz, heads)).astype(np.float32)
    for plan in plans_for(G, heads, sizes=(1, 64)):
        check_softmax_backward(csr, G, s, go, plan=plan, heads=heads, leaky=leaky)
    check_softmax_backward(csr, G, s, go, plan=fg.Plan(G, max_width=heads, segment_edges=64),
                           heads=heads, leaky=leaky, inplace=True)


@pytest.mark.parametrize("heads,dh", [(8, 16), (4, 32), (2, 64), (16, 16), (3, 16), (2, 16),
                                      (5, 20), (1, 32)])
def test_sddmm_softmax_backward(small_rmat, heads, dh):
    """The fused score gradient: one kernel for whole rows (2-16 heads of 16,
    32 or 64 features, no row cut), else the two operators; on the CSR and on
    the transposed graph with edge ids."""
    csr, G = small_rmat
    rng = np.random.default_rng(heads * 100 + dh)
    x = rng.integers(-3, 4, (csr.num_cols, heads, dh)).astype(np.float32)
    dy = rng.integers(-3, 4, (csr.num_rows, heads, dh)).astype(np.float32)
    s = (3 * rng.standard_normal((csr.nnz, heads))).astype(np.float32)
    s[rng.random(s.shape) < 0.02] = 0.0
    F = heads * dh
    for plan in (None, fg.Plan(G, F), fg.Plan(G, F, segment_edges=64)):
        for leaky in (True, False):
            check_sddmm_softmax_backward(csr, G, x, dy, s, plan=plan, leaky=leaky)
    csc = csr_to_csc(csr)
    Gt = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
    xt = rng.integers(-3, 4, (csc.num_cols, heads, dh)).astype(np.float32)
    dyt = rng.integers(-3, 4, (csc.num_rows, heads, dh)).astype(np.float32)
    check_sddmm_softmax_backward(csc, Gt, xt, dyt, s, plan=fg.Plan(Gt, F), nnz_total=csr.nnz)


def test_sddmm_softmax_backward_matches_two_calls(small_rmat):
    """With float features the fused kernel and the two separate operators
    agree closely (the same products, the sums in another order)."""
    csr, G = small_rmat
    rng = np.random.default_rng(5)
    x = rng.standard_normal((csr.num_cols, 8, 16)).astype(np.float32)
    dy = rng.standard_normal((csr.num_rows, 8, 16)).astype(np.float32)
    ts = dev((2 * rng.standard_normal((csr.nnz, 8))).astype(np.float32))
    plan = fg.Plan(G, 128)
    a = fg.edge_softmax(G, ts, plan=plan)
    fused = host(fg.gsddmm_edge_softmax_backward(G, dev(x), dev(dy), a, scores=ts, plan=plan))
    g = fg.gsddmm(G, dev(x), dev(dy), plan=plan)
    two = host(fg.edge_softmax_backward(G, a, g, scores=ts, plan=plan))
    np.testing.assert_allclose(fused, two, rtol=1e-4, atol=1e-6)
    again = host(fg.gsddmm_edge_softmax_backward(G, dev(x), dev(dy), a, scores=ts, plan=plan))
    np.testing.assert_array_equal(fused, again)  # deterministic


def test_backward_on_transposed_graph(small_rmat):
    """Max aggregation over out-edges (the CSC with edge ids): the gradient
    needs the plan's id -> position map; softmax gradient grouped by source."""
    csr, _ = small_rmat
    csc = csr_to_csc(csr)
    Gt = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
    rng = np.random.default_rng(99)
    x = rng.standard_normal((csc.num_cols, 16)).astype(np.float32)
    go = rng.standard_normal((csc.num_rows, 16)).astype(np.float32)
    w = (rng.random((csr.nnz, 2)) + 0.5).astype(np.float32)
    for seg in (0, 64):
        plan = fg.Plan(Gt, max_width=16, segment_edges=seg, max_backward=seg == 64)
        check_max_backward(csc, Gt, x, go, plan=plan, nnz_total=csr.nnz)
        check_max_backward(csc, Gt, x, go, plan=plan, edge=w, heads=2, nnz_total=csr.nnz,
                           want_edge=True)
        s = (3 * rng.standard_normal((csr.nnz, 2))).astype(np.float32)
        ge = rng.standard_normal((csr.nnz, 2)).astype(np.float32)
        check_softmax_backward(csc, Gt, s, ge, plan=plan, heads=2, nnz_total=csr.nnz)
    with pytest.raises(fg.FgError):  # no plan: no id -> position map
        fg.gspmm_max_backward(Gt, torch.zeros((csc.num_rows, 16), dtype=torch.int32,
                                              device="cuda"), dev(go))


def test_max_backward_binned_shapes():
    """The binned max backward (plan option) at the shapes that decide its
    tables: bins split over several workgroups (one hot source takes every
    row's maximum), a last tile cut short by the source count, and the shapes
    that fall back to atomics (width above the plan's, a row wider than one
    LDS tile, more tiles than the bin tables hold)."""
    rng = np.random.default_rng(2024)
    # hot source 0: 3000 rows x 16 features = 48,000 records in one bin
    n, C, F = 3000, 301, 16
    src = np.concatenate([np.zeros((n, 1), np.int64), rng.integers(1, C, (n, 4))], axis=1)
    dst = np.repeat(np.arange(n), 5)
    csr = synth.coo_to_csr(dst, src.reshape(-1), n, C)
    G = fg.Graph.from_csr(csr)
    x = rng.standard_normal((C, F)).astype(np.float32)
    x[0] = 10.0  # source 0 wins every row and feature
    go = rng.integers(-8, 9, (n, F)).astype(np.float32)
    plan = fg.Plan(G, F, max_backward=True)
    info = plan.info()
    assert info["max_backward"] == 1
    assert info["workspace_bytes"] >= 8 * n * F
    check_max_backward(csr, G, x, go, plan=plan, exact=True)
    check_max_backward(csr, G, x, rng.standard_normal((n, F)).astype(np.float32), plan=plan)
    w = rng.integers(1, 4, (csr.nnz, 1)).astype(np.float32)
    check_max_backward(csr, G, x, go, plan=plan, edge=w, want_edge=True, exact=True)
    # width above the plan's: atomics
    plan8 = fg.Plan(G, 8, max_backward=True)
    check_max_backward(csr, G, x, go, plan=plan, bwd_plan=plan8, exact=True)
    # a row wider than one LDS tile (16,384 floats): atomics
    g2 = synth.small_random_graph(np.random.default_rng(5), 12, 9, 60)
    G2 = fg.Graph.from_csr(g2)
    F2 = 16400
    x2 = rng.standard_normal((g2.num_cols, F2)).astype(np.float32)
    go2 = rng.integers(-4, 5, (g2.num_rows, F2)).astype(np.float32)
    check_max_backward(g2, G2, x2, go2, plan=fg.Plan(G2, F2, max_backward=True), exact=True)
    # 8 source rows per tile at width 2048: 70,000 sources need 8,750 tiles
    # (more than the 8,192 the tables hold): atomics; 59,999 need 7,500: binned
    for cols in (70000, 59999):
        g3 = synth.small_random_graph(np.random.default_rng(cols), 40, cols, 400)
        G3 = fg.Graph.from_csr(g3)
        x3 = rng.standard_normal((cols, 2048)).astype(np.float32)
        go3 = rng.integers(-4, 5, (40, 2048)).astype(np.float32)
        check_max_backward(g3, G3, x3, go3, plan=fg.Plan(G3, 2048, max_backward=True), exact=True)


@pytest.mark.parametrize("n,d_in,d_out", [(1, 1, 1), (17, 8, 128), (1000, 8, 33),
                                           (4099, 3, 64), (333, 130, 70), (2, 8, 512)])
def test_dense_matmul(n, d_in, d_out):
    check_dense_matmul(n, d_in, d_out, n + d_in + d_out)
    check_dense_matmul(n, d_in, d_out, n * 7 + d_out, exact=True)


@pytest.mark.parametrize("d_in,d_out", [(8, 32), (8, 128), (8, 512), (8, 6), (3, 20)])
def test_mlp_aggregate(small_rmat, d_in, d_out):
    csr, G = small_rmat
    rng = np.random.default_rng(d_in * 1000 + d_out)
    x = rng.standard_normal((csr.num_cols, d_in)).astype(np.float32)
    w = rng.standard_normal((d_in, d_out)).astype(np.float32)
    xi = rng.integers(-3, 4, (csr.num_cols, d_in)).astype(np.float32)
    wi = rng.integers(-2, 3, (d_in, d_out)).astype(np.float32)
    for plan in plans_for(G, d_out, sizes=(64,)):
        check_mlp(csr, G, x, x, w, plan=plan, square=True)
        check_mlp(csr, G, xi, xi, wi, plan=plan, square=True, exact=True)
    xd = rng.standard_normal((csr.num_rows, d_in)).astype(np.float32)
    check_mlp(csr, G, x, xd, w, plan=fg.Plan(G, d_out, segment_edges=64))


def _mlp_tie_graph(ids):
    """Rows whose messages tie only after fp32 rounding, rows whose messages
    are all 0 (ReLU), duplicate edges, an empty row.  ids: 'positions' or
    'reversed' (edge id = nnz - 1 - position, so a row's smallest id is its
    last stored edge)."""
    a, b = 2.0 ** -25, 2.0 ** -24
    xs = np.array([[a], [b], [0.5], [0.25], [2.0], [1.0]], np.float32)
    xd = np.array([[1.0], [-1.0], [0.0], [0.0], [-1.0]], np.float32)
    dst = np.array([0, 0, 1, 1, 2, 2, 2, 4, 4])
    src = np.array([0, 1, 2, 3, 1, 4, 4, 5, 2])
    csr = synth.coo_to_csr(dst, src, 5, 6)
    if ids == "reversed":
        csr = synth.CSR(5, 6, csr.indptr, csr.indices,
                        (csr.nnz - 1 - np.arange(csr.nnz)).astype(np.int32))
    return csr, xs, xd


def _mlp_rule(csr, xs, xd, w):
    """The library's rule in fp32: edges compete by P_src[u] = x_u W (raw,
    before adding P_dst[v]); the output is relu(max P_src + P_dst), taken by
    the smallest id among the edges with that largest raw value, or, when no
    message is positive (all are 0), by the row's smallest edge id."""
    ps = (xs.astype(np.float64) @ w.astype(np.float64)).astype(np.float32)
    pd = (xd.astype(np.float64) @ w.astype(np.float64)).astype(np.float32)
    out = np.zeros((csr.num_rows, w.shape[1]), np.float32)
    arg = np.full((csr.num_rows, w.shape[1]), -1, np.int32)
    for v in range(csr.num_rows):
        p = np.arange(csr.indptr[v], csr.indptr[v + 1])
        if p.size == 0:
            continue
        ids = edge_ids_of(csr, p)
        for i in range(w.shape[1]):
            raw = ps[csr.indices[p], i]
            t = raw + pd[v, i]  # fp32 sums
            if (t > 0).any():
                m = raw[t > 0].max()
                out[v, i] = np.float32(m + pd[v, i])
                arg[v, i] = ids[raw == m].min()
            else:
                arg[v, i] = ids.min()
    return out, arg


@pytest.mark.parametrize("ids", ["positions", "reversed"])
@pytest.mark.parametrize("w_row", [[1.0, 2.0, 0.5, -1.0], [1.0, 2.0, -1.0]])
def test_mlp_rounding_ties(ids, w_row):
    """One argmax rule on every path (float4 lanes with positional ids, scalar
    lanes, explicit edge ids, and the split-row merges): messages
    relu(P_src[u] + P_dst[v]) that differ only before rounding go to the
    larger P_src, and a row without a positive message reports its smallest
    edge id.  On this graph the oracle's fp64 per-edge messages pick the same
    edges, so the GPU must equal both bitwise."""
    csr, xs, xd = _mlp_tie_graph(ids)
    w = np.array([w_row], np.float32)
    G = fg.Graph.from_csr(csr)
    ro, ra = _mlp_rule(csr, xs, xd, w)
    oo, oa = O.mlp_aggregate(csr, xs, xd, w)
    np.testing.assert_array_equal(ro, oo)
    np.testing.assert_array_equal(ra, oa)
    for plan in (None, fg.Plan(G, w.shape[1], segment_edges=1)):
        say("mlp rounding ties ids=%s d_out=%d plan=%s" % (ids, w.shape[1], plan is not None))
        out, arg = fg.mlp_aggregate(G, dev(xs), dev(w), x_dst=dev(xd), plan=plan)
        np.testing.assert_array_equal(host(out).view(np.uint32), ro.view(np.uint32))
        np.testing.assert_array_equal(host(arg), ra)


def test_max_nan_messages():
    """NaN messages compete as -inf (value bits and edge ids against the
    oracle) on every max path: float4 lanes with positional ids, scalar
    lanes, explicit edge ids, weighted messages, and split rows."""
    rng = np.random.default_rng(41)
    n_rows, n_cols = 300, 200
    base = synth.small_random_graph(rng, n_rows, n_cols, 6000, 0.1)
    # rows 0..2: only NaN sources; NaN and -inf; -inf, NaN and numbers
    dst = np.concatenate([synth.csr_rows(base), [0, 0, 0, 1, 1, 2, 2, 2]])
    src = np.concatenate([base.indices, [0, 1, 2, 0, 20, 20, 0, 50]])
    csr = synth.coo_to_csr(dst, src, n_rows, n_cols)
    G = fg.Graph.from_csr(csr)
    csc = csr_to_csc(csr)
    Gt = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
    for F in (8, 5):
        x = rng.standard_normal((n_cols, F)).astype(np.float32)
        x[rng.random((n_cols, F)) < 0.3] = np.nan
        x[:20] = np.nan
        x[20:25] = -np.inf
        xt = rng.standard_normal((n_rows, F)).astype(np.float32)
        xt[rng.random((n_rows, F)) < 0.3] = np.nan
        w = rng.random(csr.nnz, dtype=np.float32)
        w[rng.random(csr.nnz) < 0.2] = 0.0  # 0 * (-inf) is NaN
        for plan in plans_for(G, F, sizes=(0, 5)):
            check_spmm(csr, G, x, plan=plan, reduce="max")
            check_spmm(csr, G, x, plan=plan, reduce="max", edge=w)
        for plan in (None, fg.Plan(Gt, F, segment_edges=5)):
            check_spmm(csc, Gt, xt, plan=plan, reduce="max", nnz_total=csr.nnz)
            check_spmm(csc, Gt, xt, plan=plan, reduce="max", edge=w, nnz_total=csr.nnz)


def test_mlp_aggregate_transposed_and_empty(small_rmat):
    csr, _ = small_rmat
    csc = csr_to_csc(csr)
    Gt = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
    rng = np.random.default_rng(5)
    x = rng.integers(-3, 4, (csc.num_cols, 8)).astype(np.float32)
    w = rng.integers(-2, 3, (8, 16)).astype(np.float32)
    xf = rng.standard_normal((csc.num_cols, 8)).astype(np.float32)
    wf = rng.standard_normal((8, 16)).astype(np.float32)
    for plan in (None, fg.Plan(Gt, 16, segment_edges=64)):
        check_mlp(csc, Gt, x, x, w, plan=plan, exact=True, square=True)
        # float inputs through explicit edge ids (messages masked in the loop)
        check_mlp(csc, Gt, xf, xf, wf, plan=plan, square=True)
        check_mlp(csc, Gt, xf[:, :7].copy(), xf[:, :7].copy(), wf[:7, :7].copy(), plan=None,
                  square=True)  # odd width: scalar lanes
    noedge = synth.CSR(3, 5, np.zeros(4, np.int32), np.zeros(0, np.int32))
    G0 = fg.Graph.from_csr(noedge)
    o, a = fg.mlp_aggregate(G0, dev(np.ones((5, 8), np.float32)), dev(np.ones((8, 4), np.float32)),
                            x_dst=dev(np.ones((3, 8), np.float32)))
    assert np.all(host(o) == 0) and np.all(host(a) == -1)


@pytest.mark.parametrize("d", [4, 16, 33, 64, 128, 512, 1024, 1040])
def test_sddmm_edge_softmax(small_rmat, d):
    csr, G = small_rmat
    rng = np.random.default_rng(d + 5)
    x = (rng.standard_normal((csr.num_cols, d)) / math.sqrt(d) * 3).astype(np.float32)
    xd = (rng.standard_normal((csr.num_rows, d)) / math.sqrt(d) * 3).astype(np.float32)
    for plan in plans_for(G, d, sizes=(1, 64)):
        check_sddmm_softmax(csr, G, x, xd, plan=plan)
    check_sddmm_softmax(csr, G, x, xd, plan=fg.Plan(G, d, segment_edges=64), leaky=False)


def test_sddmm_edge_softmax_heads_and_transposed(small_rmat):
    csr, G = small_rmat
    rng = np.random.default_rng(3)
    x = rng.standard_normal((csr.num_cols, 8, 16)).astype(np.float32) * 0.5
    check_sddmm_softmax(csr, G, x, x, heads=8, plan=fg.Plan(G, 128, segment_edges=64))
    csc = csr_to_csc(csr)
    Gt = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
    y = rng.standard_normal((csc.num_cols, 32)).astype(np.float32) * 0.3
    yd = rng.standard_normal((csc.num_rows, 32)).astype(np.float32) * 0.3
    for plan in (None, fg.Plan(Gt, 32, segment_edges=64)):
        check_sddmm_softmax(csc, Gt, y, yd, plan=plan, nnz_total=csr.nnz)


def test_gat_fused_unsupported_shape_raises(small_rmat):
    csr, G = small_rmat
    x = dev(np.ones((csr.num_cols, 3, 12), np.float32))
    with pytest.raises(fg.FgError) as ei:
        fg.gat_aggregate(G, x)
    assert ei.value.status == fg.FG_ERR_UNSUPPORTED


def test_transposed_graph_with_edge_ids(small_rmat):
    csr, _ = small_rmat
    csc = csr_to_csc(csr)
    G = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
    rng = np.random.default_rng(3)
    y = rng.standard_normal((csc.num_cols, 24)).astype(np.float32)
    x = rng.standard_normal((csc.num_rows, 24)).astype(np.float32)
    wgt = rng.random((csr.nnz, 1), dtype=np.float32)
    # default plan: short rows of the softmax are packed four to a wavefront
    for plan in plans_for(G, 24, sizes=(0, 16)):
        check_spmm(csc, G, y, plan=plan, nnz_total=csr.nnz)
        check_spmm(csc, G, y, plan=plan, edge=wgt, nnz_total=csr.nnz)
        check_spmm(csc, G, y, plan=plan, reduce="max", nnz_total=csr.nnz)
        check_sddmm(csc, G, y, x, plan=plan, nnz_total=csr.nnz)
        check_softmax(csc, G, rng.standard_normal(csr.nnz).astype(np.float32), plan=plan,
                      nnz_total=csr.nnz)
    # per-head edge values through edge ids (staged a batch ahead), 4 heads of 8
    y4 = rng.standard_normal((csc.num_cols, 4, 8)).astype(np.float32)
    w4 = rng.random((csr.nnz, 4), dtype=np.float32)
    for plan in plans_for(G, 32, sizes=(0, 16)):
        check_spmm(csc, G, y4, plan=plan, edge=w4, heads=4, nnz_total=csr.nnz)
        check_spmm(csc, G, y4, plan=plan, edge=w4, heads=4, reduce="max", nnz_total=csr.nnz)


def test_edge_cases():
    # no rows at all
    empty = synth.CSR(0, 5, np.zeros(1, np.int32), np.zeros(0, np.int32))
    G = fg.Graph.from_csr(empty)
    out = fg.gspmm(G, dev(np.ones((5, 4), np.float32)))
    assert out.shape == (0, 4)
    # rows but no edges: sum 0, max 0 / -1, sddmm / softmax write nothing
    noedge = synth.CSR(3, 5, np.zeros(4, np.int32), np.zeros(0, np.int32))
    G = fg.Graph.from_csr(noedge)
    for plan in (None, fg.Plan(G, 8, 4)):
        o = host(fg.gspmm(G, dev(np.ones((5, 8), np.float32)), plan=plan))
        assert np.all(o == 0)
        o, a = fg.gspmm(G, dev(np.ones((5, 8), np.float32)), reduce="max", plan=plan)
        assert np.all(host(o) == 0) and np.all(host(a) == -1)
        s = fg.gsddmm(G, dev(np.ones((5, 8), np.float32)), dev(np.ones((3, 8), np.float32)),
                      plan=plan)
        assert s.numel() == 0
    # signed zeros, -inf rows, duplicate edges, single-edge rows
    g = synth.CSR(4, 4, np.array([0, 2, 4, 6, 7], np.int32),
                  np.array([0, 1, 1, 0, 2, 3, 1], np.int32))
    x = np.array([[-0.0, 1.0], [0.0, 1.0], [-np.inf, -np.inf], [-np.inf, 5.0]], np.float32)
    G = fg.Graph.from_csr(g)
    for plan in (None, fg.Plan(G, 2, 1)):
        check_spmm(g, G, x, plan=plan, reduce="max")
    dup = synth.CSR(2, 3, np.array([0, 5, 6], np.int32), np.array([1, 1, 1, 2, 2, 0], np.int32))
    G = fg.Graph.from_csr(dup)
    xi = np.array([[1, 2, 3, 4], [5, 5, 5, 5], [5, 0, 5, 0]], np.float32)
    for plan in (None, fg.Plan(G, 4, 2), fg.Plan(G, 4, 2, max_backward=True)):
        check_spmm(dup, G, xi, plan=plan, reduce="max")
        check_spmm(dup, G, xi, plan=plan, exact=True)
        s = check_sddmm(dup, G, xi, xi[:2], plan=plan, exact=True)
        a = host(fg.edge_softmax(G, dev(np.full(6, 3.0, np.float32)), plan=plan))
        np.testing.assert_allclose(a, [0.2] * 5 + [1.0], rtol=1e-6)
        del s
        # gradients through duplicate edges and ties: the smallest edge id takes it
        check_max_backward(dup, G, xi, np.arange(8, dtype=np.float32).reshape(2, 4), plan=plan,
                           exact=True)
        check_max_backward(dup, G, xi, np.ones((2, 4), np.float32), plan=plan,
                           edge=np.array([1, 2, 1, 2, 1, 1], np.float32), want_edge=True,
                           exact=True)
        check_softmax_backward(dup, G, np.full(6, 3.0, np.float32),
                               np.arange(6, dtype=np.float32), plan=plan)
        # fused score gradient (2 heads of 16) through duplicates and equal scores
        xh = np.arange(96, dtype=np.float32).reshape(3, 2, 16) % 5 - 2
        dyh = np.arange(64, dtype=np.float32).reshape(2, 2, 16) % 3 - 1
        check_sddmm_softmax_backward(dup, G, xh, dyh, np.full((6, 2), 3.0, np.float32),
                                     plan=None if plan is None else fg.Plan(
                                         G, 32, 2 if plan.info()["max_backward"] else 0))
    # backward without edges: gradients all zero, softmax gradient writes nothing
    G = fg.Graph.from_csr(noedge)
    for plan in (None, fg.Plan(G, 8, 4), fg.Plan(G, 8, 4, max_backward=True)):
        gs = fg.gspmm_max_backward(G, torch.full((3, 8), -1, dtype=torch.int32, device="cuda"),
                                   dev(np.ones((3, 8), np.float32)), plan=plan)
        assert gs.shape == (5, 8) and np.all(host(gs) == 0)
        ds = fg.edge_softmax_backward(G, dev(np.zeros(0, np.float32)),
                                      dev(np.zeros(0, np.float32)),
                                      scores=dev(np.zeros(0, np.float32)), plan=plan)
        assert ds.numel() == 0
        ds = fg.gsddmm_edge_softmax_backward(
            G, dev(np.ones((5, 2, 4), np.float32)), dev(np.ones((3, 2, 4), np.float32)),
            dev(np.zeros((0, 2), np.float32)), scores=dev(np.zeros((0, 2), np.float32)))
        assert ds.numel() == 0


def _blocked_graph(rng, n, deg_hi):
    """Rows in blocks of 40 drawing sources from one block of 64 ids
    (neighbouring rows share sources), degrees 1..deg_hi."""
    deg = rng.integers(1, deg_hi + 1, n)
    dst = np.repeat(np.arange(n), deg)
    base = (dst // 40 * 64) % max(n - 64, 1)
    src = np.minimum(base + rng.integers(0, 64, dst.size), n - 1)
    return synth.coo_to_csr(dst, src, n, n)


_WIDTHS = (1, 2, 3, 4, 8, 12, 16, 20, 32, 48, 64, 96, 128, 160, 256, 300, 512, 1024, 1040)


@pytest.mark.parametrize("seed", range(160))
def test_random_configurations(seed):
    """Seeded sweep over graph shapes (uniform, power-law with hubs, blocked
    communities, bipartite; sometimes transposed with edge ids), widths,
    heads, operators and plan options (segment length, source slabs, item
    order): each case against the oracle on every row."""
    rng = np.random.default_rng(1000 + seed)
    kind = ("uniform", "rmat", "blocked", "bipartite")[seed % 4]
    n = int(rng.integers(2, 2500))
    if kind == "uniform":
        csr = synth.uniform_graph(rng, n, int(rng.integers(0, 40 * n)))
    elif kind == "bipartite":  # sources and destinations of different counts
        m = int(rng.integers(1, 3000))
        e = int(rng.integers(0, 40 * n))
        csr = synth.coo_to_csr(rng.integers(0, n, e), rng.integers(0, m, e), n, m)
    elif kind == "rmat":
        scale = max(1, int(np.ceil(np.log2(n))))
        csr = synth.rmat_graph(np.random.SeedSequence(seed), rng, scale, n,
                               int(rng.integers(1, 30 * n)), workers=1)
    else:
        csr = _blocked_graph(rng, n, int(rng.integers(1, 120)))
    F = int(rng.choice(_WIDTHS))
    heads = int(rng.choice([h for h in (1, 2, 4, 8, 16) if F % h == 0]))
    nnz_total = None
    g = csr
    if seed % 5 == 3:  # the transposed graph with edge ids
        g, nnz_total = csr_to_csc(csr), csr.nnz
    square = g.num_rows == g.num_cols
    x = rng.standard_normal((g.num_cols, F)).astype(np.float32)
    xd = rng.standard_normal((g.num_rows, F)).astype(np.float32)
    if heads > 1:
        x = x.reshape(g.num_cols, heads, F // heads)
        xd = xd.reshape(g.num_rows, heads, F // heads)
    G = fg.Graph.from_csr(g, nnz_total=nnz_total or 0)
    if rng.random() < 0.2:
        plan = None
    else:
        seg = int(rng.choice([0, 1, 7, 64, 512]))
        slab = int(rng.choice([0, -1, -2, 37, 500]))
        min_deg = int(rng.choice([0, 1, 16]))
        order = int(rng.integers(0, 3))
        if order == 1 and seed % 3 == 0:
            order = 3  # die-banded (drawn this way to keep every seed's other draws)
        plan = fg.Plan(G, max(F, heads, 1), segment_edges=seg, source_slab_rows=slab,
                       partition_min_degree=min_deg, item_order=order,
                       max_backward=seed % 2 == 1)
        say("plan", plan.info())
    ops = rng.choice(["sum", "mul", "max", "sddmm", "softmax", "softmax_bwd", "max_bwd", "gat",
                      "mlp", "sddmm_softmax", "sddmm_softmax_bwd"], size=3, replace=False)
    say("seed", seed, kind, "n", n, "nnz", g.nnz, "F", F, "heads", heads, "ops", list(ops))
    _check_ops(rng, ops, g, G, x, xd, plan, heads, nnz_total)


@pytest.mark.parametrize("seed", range(40))
def test_random_configurations_long_rows(seed):
    """Seeded sweep over graphs whose rows average 64 to 400 edges (uniform,
    power-law with hubs, blocked communities; sometimes transposed with edge
    ids), so that the gather kernels take their 256-edge batches, at widths
    of one to sixteen lane groups, with heads, operators and plan options
    (segment length, source slabs, item order, mid-length cut): each case
    against the oracle on every row."""
    rng = np.random.default_rng(5000 + seed)
    kind = ("uniform", "rmat", "blocked")[seed % 3]
    n = int(rng.integers(64, 1500))
    avg = int(rng.integers(64, 400))
    if kind == "uniform":
        csr = synth.uniform_graph(rng, n, n * avg)
    elif kind == "rmat":
        scale = max(1, int(np.ceil(np.log2(n))))
        csr = synth.rmat_graph(np.random.SeedSequence(5000 + seed), rng, scale, n, n * avg,
                               workers=1)
    else:
        csr = _blocked_graph(rng, n, 2 * avg)
    F = int(rng.choice((16, 20, 32, 48, 64, 96, 100, 128, 256)))
    heads = int(rng.choice([h for h in (1, 2, 4, 8) if F % h == 0]))
    nnz_total = None
    g = csr
    if seed % 5 == 2:  # the transposed graph with edge ids
        g, nnz_total = csr_to_csc(csr), csr.nnz
    x = rng.standard_normal((g.num_cols, F)).astype(np.float32)
    xd = rng.standard_normal((g.num_rows, F)).astype(np.float32)
    if heads > 1:
        x = x.reshape(g.num_cols, heads, F // heads)
        xd = xd.reshape(g.num_rows, heads, F // heads)
    G = fg.Graph.from_csr(g, nnz_total=nnz_total or 0)
    if rng.random() < 0.2:
        plan = None
    else:
        plan = fg.Plan(G, F, segment_edges=int(rng.choice([0, 100, 512, 2048, 8192])),
                       source_slab_rows=int(rng.choice([0, -2, 300])),
                       item_order=int(rng.choice([0, 1, 3])),
                       band_row_edges=int(rng.choice([0, -1, 100])))
        say("plan", plan.info())
    ops = rng.choice(["sum", "mul", "max", "sddmm", "softmax", "gat", "mlp", "sddmm_softmax"],
                     size=3, replace=False)
    say("seed", seed, kind, "n", n, "nnz", g.nnz, "F", F, "heads", heads, "ops", list(ops))
    _check_ops(rng, ops, g, G, x, xd, plan, heads, nnz_total)


def _check_ops(rng, ops, g, G, x, xd, plan, heads, nnz_total):
    """Each of ops on graph g (G on the device) against the oracle on every
    row; draws its extra inputs from rng."""
    n, F = g.num_rows, int(np.prod(x.shape[1:]))
    square = g.num_rows == g.num_cols
    nt = nnz_total or g.nnz
    for op in ops:
        if op == "sum":
            check_spmm(g, G, x, plan=plan, heads=heads, nnz_total=nnz_total)
        elif op == "mul":
            w = rng.random((nt, heads), dtype=np.float32)
            check_spmm(g, G, x, plan=plan, edge=w, heads=heads, nnz_total=nnz_total)
        elif op == "max":
            check_spmm(g, G, x, plan=plan, reduce="max", heads=heads, nnz_total=nnz_total)
        elif op == "sddmm":
            check_sddmm(g, G, x, xd, plan=plan, heads=heads, nnz_total=nnz_total)
        elif op == "softmax":
            sc = (rng.standard_normal((nt, heads)) * 3).astype(np.float32)
            check_softmax(g, G, sc, plan=plan, heads=heads, nnz_total=nnz_total)
        elif op == "softmax_bwd":
            sc = (rng.standard_normal((nt, heads)) * 3).astype(np.float32)
            go = rng.standard_normal((nt, heads)).astype(np.float32)
            check_softmax_backward(g, G, sc, go, plan=plan, heads=heads, nnz_total=nnz_total)
        elif op == "max_bwd" and nnz_total is None:
            go = rng.integers(-4, 5, (g.num_rows, F)).astype(np.float32).reshape(
                (g.num_rows,) + x.shape[1:])
            check_max_backward(g, G, x, go, plan=plan, heads=heads, exact=True)
        elif op == "gat" and nnz_total is None and square:
            dh = F // heads
            if dh % 4 == 0 and (dh // 4) & (dh // 4 - 1) == 0 and F <= 256:
                check_gat(g, G, x.reshape(n, heads, dh), plan=plan, heads=heads)
            else:
                with pytest.raises(fg.FgError):
                    fg.gat_aggregate(G, dev(x.reshape(n, heads, dh)), plan=plan)
        elif op == "mlp" and nnz_total is None:
            d_in = int(rng.choice([1, 3, 8]))
            xi = rng.integers(-3, 4, (g.num_cols, d_in)).astype(np.float32)
            xj = rng.integers(-3, 4, (g.num_rows, d_in)).astype(np.float32)
            wi = rng.integers(-2, 3, (d_in, F)).astype(np.float32)
            check_mlp(g, G, xi, xj, wi, plan=plan, exact=True, square=False)
        elif op == "sddmm_softmax":
            check_sddmm_softmax(g, G, x, xd, plan=plan, heads=heads, nnz_total=nnz_total)
        elif op == "sddmm_softmax_bwd":
            dh = F // heads
            xi = rng.integers(-3, 4, (g.num_cols, heads, dh)).astype(np.float32)
            di = rng.integers(-3, 4, (g.num_rows, heads, dh)).astype(np.float32)
            sc = (rng.standard_normal((nt, heads)) * 3).astype(np.float32)
            check_sddmm_softmax_backward(g, G, xi, di, sc, plan=plan, nnz_total=nnz_total)


def _odd(a=None, shape=None, dtype=torch.float32):
    """A contiguous device tensor that starts 4 bytes past a 16-byte boundary."""
    shape = a.shape if a is not None else shape
    n = int(np.prod(shape))
    buf = torch.zeros(n + 4, dtype=dtype, device="cuda")
    t = buf[1:1 + n].view(shape)
    assert t.data_ptr() % 16 == 4
    if a is not None:
        t.copy_(torch.from_numpy(np.ascontiguousarray(a)))
    return t


def test_misaligned_pointers(small_rmat):
    """Every array 4 bytes off a 16-byte boundary: the kernels' float4 paths
    must step aside for the scalar ones and give the oracle's results."""
    csr, G = small_rmat
    n, e = csr.num_rows, csr.nnz
    rng = np.random.default_rng(23)
    plan = fg.Plan(G, 128)
    x = rng.standard_normal((n, 128)).astype(np.float32)
    x8 = x.reshape(n, 8, 16)
    w8 = rng.random((e, 8), dtype=np.float32)
    deg = csr.degrees()[:, None]
    # gSpMM: copy + sum, per-head weights, max + argmax
    out = _odd(shape=(n, 128))
    fg.gspmm(G, _odd(x), plan=plan, out=out)
    ro, nrm = O.gspmm(csr, x, with_norm=True)
    assert_close_sum(host(out), ro.astype(np.float64), nrm, deg)
    out8 = _odd(shape=(n, 8, 16))
    fg.gspmm(G, _odd(x8), _odd(w8), msg="src_mul_edge", plan=plan, out=out8)
    ro, nrm = O.gspmm(csr, x, msg=O.MSG_SRC_MUL_EDGE, heads=8, edge_val=w8, with_norm=True)
    assert_close_sum(host(out8).reshape(n, 128), ro.astype(np.float64), nrm, deg)
    arg = _odd(shape=(n, 128), dtype=torch.int32)
    fg.gspmm(G, _odd(x), reduce="max", plan=plan, out=out, arg=arg)
    rm, ra = O.gspmm(csr, x, red=O.RED_MAX)
    np.testing.assert_array_equal(host(out).view(np.uint32), rm.view(np.uint32))
    np.testing.assert_array_equal(host(arg), ra)
    # gSDDMM per head
    sc = _odd(shape=(e, 8))
    fg.gsddmm(G, _odd(x8), _odd(x8), plan=plan, out=sc)
    rs, nrm = O.gsddmm(csr, x, x, heads=8, with_norm=True)
    assert_close_sum(host(sc), rs.astype(np.float64), nrm, 16)
    # edge softmax and its gradient, on the oracle's scores
    a = _odd(shape=(e, 8))
    fg.edge_softmax(G, _odd(rs), leaky=True, slope=0.2, plan=plan, out=a)
    ra = O.edge_softmax(csr, rs, heads=8, leaky=True, slope=0.2)
    assert_close_softmax(host(a), ra, np.repeat(csr.degrees(), csr.degrees())[:, None])
    ga = rng.standard_normal((e, 8)).astype(np.float32)
    ds = _odd(shape=(e, 8))
    fg.edge_softmax_backward(G, _odd(ra), _odd(ga), scores=_odd(rs), leaky=True, slope=0.2,
                             plan=plan, grad_scores=ds)
    rd, scale = O.edge_softmax_backward(csr, rs, ga, heads=8, leaky=True, slope=0.2,
                                        with_scale=True)
    bound = 1e-5 * np.sqrt(np.repeat(np.maximum(csr.degrees(), 1), csr.degrees()))[:, None] * scale
    assert (np.abs(host(ds).astype(np.float64) - rd) <= bound + 1e-12).all()
    # fused SDDMM + softmax, one head
    s1, a1 = _odd(shape=(e,)), _odd(shape=(e,))
    fg.gsddmm_edge_softmax(G, _odd(x), _odd(x), plan=plan, scores=s1, out=a1)
    r1, nrm = O.gsddmm(csr, x, x, with_norm=True)
    assert_close_sum(host(s1)[:, None], r1.astype(np.float64), nrm, 128)
    nz = csr.degrees() > 0
    rsum = np.add.reduceat(host(a1).astype(np.float64), csr.indptr[:-1][nz])
    np.testing.assert_allclose(rsum, 1.0, atol=1e-5 * math.sqrt(csr.degrees().max()))
    # the fused attention layer needs 16-byte aligned rows and says so
    with pytest.raises(fg.FgError):
        fg.gat_aggregate(G, _odd(x8), _odd(x8), plan=plan, out=_odd(shape=(n, 8, 16)))


def test_determinism_and_plan_independence(small_rmat):
    csr, G = small_rmat
    x = np.random.default_rng(9).standard_normal((csr.num_cols, 128)).astype(np.float32)
    tx = dev(x)
    plan = fg.Plan(G, 128, 32, source_slab_rows=250, partition_min_degree=1)
    assert plan.info()["num_partitioned_rows"] > 0
    a1 = host(fg.gspmm(G, tx, plan=plan))
    a2 = host(fg.gspmm(G, tx, plan=plan))
    np.testing.assert_array_equal(a1.view(np.uint32), a2.view(np.uint32))
    m1, i1 = (host(t) for t in fg.gspmm(G, tx, reduce="max", plan=plan))
    m0, i0 = (host(t) for t in fg.gspmm(G, tx, reduce="max"))
    np.testing.assert_array_equal(m1.view(np.uint32), m0.view(np.uint32))
    np.testing.assert_array_equal(i1, i0)
    s1 = host(fg.gsddmm(G, tx, tx[: csr.num_rows].contiguous(), plan=plan))
    s2 = host(fg.gsddmm(G, tx, tx[: csr.num_rows].contiguous()))
    np.testing.assert_array_equal(s1.view(np.uint32), s2.view(np.uint32))


def test_die_banded_order_gives_identical_results(small_rmat):
    """Without the extra cut of mid-length rows (band_row_edges = -1) the
    die-banded gather order runs the same pieces with the same slots as
    longest-first order, so every result is bitwise the same."""
    csr, G = small_rmat
    rng = np.random.default_rng(12)
    x = rng.standard_normal((csr.num_cols, 64)).astype(np.float32)
    w = rng.random(csr.nnz, dtype=np.float32)
    p1 = fg.Plan(G, 64, segment_edges=16, item_order=1)
    p3 = fg.Plan(G, 64, segment_edges=16, item_order=3, band_row_edges=-1)
    assert p3.info()["item_order"] == 3 and p3.info()["num_segments"] > p1.info()["num_segments"]
    tx, tw = dev(x), dev(w)
    for name, f in (("mul_sum", lambda p: fg.gspmm(G, tx, tw, msg="src_mul_edge", plan=p)),
                    ("max", lambda p: fg.gspmm(G, tx, reduce="max", plan=p)[0]),
                    ("sddmm", lambda p: fg.gsddmm(G, tx, tx, plan=p))):
        say("die-banded vs longest first:", name)
        np.testing.assert_array_equal(host(f(p3)).view(np.uint32), host(f(p1)).view(np.uint32))
    check_spmm(csr, G, x, plan=p3, edge=w)


def test_plan_bound_to_its_graph(small_rmat):
    csr, G = small_rmat
    other = fg.Graph.from_csr(csr)  # same structure, different device arrays
    plan = fg.Plan(G, 16)
    x = dev(np.ones((csr.num_cols, 16), np.float32))
    with pytest.raises(fg.FgError):
        fg.gspmm(other, x, plan=plan)
    with pytest.raises(fg.FgError):
        fg.gspmm(G, dev(np.ones((csr.num_cols, 32), np.float32)), plan=plan)  # too wide


def test_plan_checksum_after_in_place_edit():
    """A plan is not reused after its graph's indptr was edited in place: the
    binding refuses it (modification counters), fg_plan_validate sees the
    changed checksum, and restoring indptr makes the plan valid again."""
    csr = make_config("tiny_uniform_1k").csr
    G = fg.Graph.from_csr(csr)
    plan = fg.Plan(G, 32, segment_edges=5)
    assert plan.info()["indptr_checksum"] == fg.indptr_checksum(csr.indptr)
    x = np.random.default_rng(9).standard_normal((csr.num_cols, 32)).astype(np.float32)
    plan.validate()
    say("plan checksum: edit indptr in place")
    old = int(csr.indptr[1])
    G.indptr[1] = old - 1  # one edge moves from row 0 to row 1: same shape, same nnz
    with pytest.raises(ValueError, match="modified in place"):
        fg.gspmm(G, dev(x), plan=plan)
    with pytest.raises(fg.FgError):
        plan.validate()
    st = fg._lib.fg_plan_validate(plan.handle, ctypes.byref(G._c), None, fg._stream())
    assert st == fg.FG_ERR_INVALID_ARG
    G.indptr[1] = old
    plan.validate()  # contents match again: accepted, counters re-recorded
    check_spmm(csr, G, x, plan=plan)
    # another graph of the same shape at another address is refused by pointer
    other = fg.Graph.from_csr(csr)
    assert fg._lib.fg_plan_validate(plan.handle, ctypes.byref(other._c), None,
                                    fg._stream()) == fg.FG_ERR_INVALID_ARG
    plan.close()


# ----------------------------------------------------------------------------
# the five named workloads at full size (sampled rows against the oracle)
# ----------------------------------------------------------------------------


@pytest.mark.parametrize("d", [32, 64, 128, 256, 512])
def test_uniform_deg100_full(d):
    w = make_config("uniform_deg100_100k", d=d)
    csr = w.csr
    G = fg.Graph.from_csr(csr)
    x = w.arrays["x"]
    rows = sample_rows(csr, 3000, d)
    plan = fg.Plan(G, d)
    check_spmm(csr, G, x, rows=rows, plan=plan)
    check_sddmm(csr, G, x, x, rows=rows, plan=plan)
    # source slabs: at d = 128 every row is cut by default (spread gathers) and
    # with -1; at the other widths rows of 100 edges stay whole
    aplan = fg.Plan(G, d, source_slab_rows=-1)
    assert (aplan.info()["num_partitioned_rows"] == csr.num_rows) == (d == 128)
    assert plan.info()["num_partitioned_rows"] == aplan.info()["num_partitioned_rows"]
    if d == 128:
        nplan = fg.Plan(G, d, source_slab_rows=-2)
        assert nplan.info()["num_partitioned_rows"] == 0
        check_spmm(csr, G, x, rows=rows, plan=nplan)
        check_sddmm(csr, G, x, x, rows=rows, plan=nplan)
    # property over every row: all-ones features sum to the in-degree (100)
    o = host(fg.gspmm(G, dev(np.ones((csr.num_cols, d), np.float32)), plan=plan))
    assert np.all(o == 100.0)


@pytest.fixture(scope="module")
def rmat_full():
    w = make_config("rmat_233k_115m")
    return w, fg.Graph.from_csr(w.csr)


@pytest.mark.slow
def test_rmat_233k_full(rmat_full):
    w, G = rmat_full
    csr = w.csr
    x, wgt = w.arrays["x"], w.arrays["w"]
    plan = fg.Plan(G, 128)
    info = plan.info()
    say("plan", info)
    assert info["num_split_rows"] > 0
    # source-partitioned gather schedule of the same graph (automatic slab size)
    pplan = fg.Plan(G, 128, source_slab_rows=-1)
    assert pplan.info()["num_partitioned_rows"] > 0
    rows = sample_rows(csr, 2000, 3)
    check_spmm(csr, G, x, rows=rows, plan=plan, edge=wgt)
    check_spmm(csr, G, x, rows=rows, plan=plan, reduce="max")
    check_sddmm(csr, G, x, x, rows=rows, plan=plan)
    # softmax on seeded scores of the SDDMM's scale (N(0, d)), the same array on both sides
    s_syn = (np.random.default_rng(31).standard_normal(csr.nnz, dtype=np.float32)
             * np.float32(math.sqrt(128)))
    check_softmax(csr, G, s_syn, rows=rows, plan=plan)
    # SDDMM and softmax in one call, in the benchmark's launch configuration
    # (long items: the two kernels), and as the fused kernel (64-edge items)
    check_sddmm_softmax(csr, G, x, x, rows=rows, plan=plan)
    check_sddmm_softmax(csr, G, x, x, rows=rows, plan=fg.Plan(G, 128, segment_edges=64))
    check_spmm(csr, G, x, rows=rows, plan=pplan, edge=wgt)
    check_spmm(csr, G, x, rows=rows, plan=pplan, reduce="max")
    check_sddmm(csr, G, x, x, rows=rows, plan=pplan)
    o = host(fg.gspmm(G, dev(np.ones((csr.num_cols, 128), np.float32)), plan=plan))
    np.testing.assert_array_equal(o[:, 0], csr.degrees().astype(np.float32))
    np.testing.assert_array_equal(o[:, 127], csr.degrees().astype(np.float32))


@pytest.mark.slow
def test_rmat_233k_max_backward_full(rmat_full):
    """GraphSage-max gradient on the whole power-law graph in the benchmark's
    launch configuration; integer upstream gradients make the sums exact, so
    the whole [N, 128] gradient must equal the oracle's bit for bit."""
    w, G = rmat_full
    csr = w.csr
    go = np.random.default_rng(8).integers(-8, 9, (csr.num_rows, 128)).astype(np.float32)
    for binned in (False, True):
        plan = fg.Plan(G, 128, max_backward=binned)
        assert plan.info()["max_backward"] == int(binned)
        check_max_backward(csr, G, w.arrays["x"], go, plan=plan, exact=True)
        plan.close()


@pytest.mark.slow
def test_rmat_233k_mlp_full(rmat_full):
    """MLP aggregation (d_in 8 -> d_out 128) on the whole power-law graph in
    the benchmark's configuration, checked on sampled rows."""
    w_, G = rmat_full
    csr = w_.csr
    rng = np.random.default_rng(21)
    x = rng.standard_normal((csr.num_cols, 8)).astype(np.float32)
    w = rng.standard_normal((8, 128)).astype(np.float32)
    rows = sample_rows(csr, 300, 22)
    check_mlp(csr, G, x, x, w, rows=rows, plan=fg.Plan(G, 128), square=True)


@pytest.mark.slow
def test_clustered_gat_layer_full():
    w = make_config("clustered_133k_deg300")
    csr = w.csr
    G = fg.Graph.from_csr(csr)
    x = w.arrays["x"]
    plan = fg.Plan(G, 128)
    rows = sample_rows(csr, 1500, 4)
    check_sddmm(csr, G, x, x, rows=rows, plan=plan, heads=8)
    # softmax and weighted aggregation on seeded scores of the SDDMM's scale
    # (N(0, dh)); the aggregation's weights are the oracle's softmax of them
    s_syn = (np.random.default_rng(32).standard_normal((csr.nnz, 8), dtype=np.float32)
             * np.float32(4.0))
    a = check_softmax(csr, G, s_syn, rows=rows, plan=plan, heads=8)
    a_ref = O.edge_softmax(csr, s_syn, heads=8, leaky=True, slope=0.2)
    check_spmm(csr, G, x, rows=rows, plan=plan, edge=a_ref, heads=8)
    # softmax rows sum to one for every row and head
    rs = np.add.reduceat(host(a).astype(np.float64), csr.indptr[:-1], axis=0)
    np.testing.assert_allclose(rs, 1.0, atol=1e-5 * math.sqrt(300))
    # the fused layer on the same graph
    check_gat(csr, G, x, rows=rows, plan=plan, heads=8)
    # gradient of the softmax (upstream gradient of the attention weights)
    ga = np.random.default_rng(9).standard_normal((csr.nnz, 8)).astype(np.float32)
    check_softmax_backward(csr, G, s_syn, ga, rows=rows, plan=plan, heads=8)


@pytest.mark.slow
def test_clustered_gat_backward_full():
    """Backward of the attention layer on the whole clustered graph in the
    benchmark's launch configuration: per-head aggregations on the transposed
    graph, which read the edge values through edge ids, and the per-head
    gradient SDDMM."""
    w = make_config("clustered_133k_deg300")
    csr = w.csr
    csc = csr_to_csc(csr)
    G = fg.Graph.from_csr(csr)
    Gt = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
    x = w.arrays["x"]
    n, H, dh = x.shape
    gy = np.random.default_rng(12).standard_normal((n, H, dh)).astype(np.float32)
    a = O.edge_softmax(csr, (np.random.default_rng(33).standard_normal((csr.nnz, H),
                                                                       dtype=np.float32)
                             * np.float32(4.0)), heads=H, leaky=True, slope=0.2)
    ds = np.random.default_rng(34).standard_normal((csr.nnz, H)).astype(np.float32) * 1e-2
    P, Pt = fg.Plan(G, H * dh), fg.Plan(Gt, H * dh)
    rows = sample_rows(csr, 1000, 13)
    rows_t = sample_rows(csc, 1000, 14)
    check_spmm(csc, Gt, gy, rows=rows_t, plan=Pt, edge=a, heads=H, nnz_total=csr.nnz)
    check_spmm(csc, Gt, x, rows=rows_t, plan=Pt, edge=ds, heads=H, nnz_total=csr.nnz)
    check_spmm(csc, Gt, x, rows=rows_t, plan=None, edge=ds, heads=H, nnz_total=csr.nnz)
    check_spmm(csr, G, x, rows=rows, plan=P, edge=ds, heads=H)
    check_sddmm(csr, G, x, gy, rows=rows, plan=P, heads=H)
    # the score gradient in one call (fused kernel: no row of this graph is
    # cut), with small-integer features so that the dot products are exact
    rng = np.random.default_rng(35)
    xi = rng.integers(-3, 4, x.shape).astype(np.float32)
    gi = rng.integers(-3, 4, gy.shape).astype(np.float32)
    s = (4 * rng.standard_normal((csr.nnz, H))).astype(np.float32)
    check_sddmm_softmax_backward(csr, G, xi, gi, s, plan=P, rows=rows)


@pytest.mark.slow
@pytest.mark.parametrize("d", [32, 128])
def test_rand_100k_full(d):
    """The two-degree-class graph (20K vertices at mean in-degree 2000, 80K
    at 100) under the default and the source-partitioned schedules."""
    w = make_config("rand_100k_48m", d=d)
    csr = w.csr
    G = fg.Graph.from_csr(csr)
    x = w.arrays["x"]
    rows = sample_rows(csr, 600, 15 + d)
    plan = fg.Plan(G, d)
    # automatic slabs at d = 128; at d = 32 the features fit the dies' L2s and
    # the automatic rule leaves the graph whole, so slabs are given
    pplan = fg.Plan(G, d, source_slab_rows=-1 if d >= 128 else 4096)
    assert pplan.info()["num_partitioned_rows"] > 0
    assert fg.Plan(G, 32, source_slab_rows=-1).info()["num_partitioned_rows"] == 0
    for p in (plan, pplan):
        check_spmm(csr, G, x, rows=rows, plan=p)
        check_spmm(csr, G, x, rows=rows, plan=p, reduce="max")
        check_sddmm(csr, G, x, x, rows=rows, plan=p)
    o = host(fg.gspmm(G, dev(np.ones((csr.num_cols, d), np.float32)), plan=pplan))
    np.testing.assert_array_equal(o[:, -1], csr.degrees().astype(np.float32))


@pytest.mark.slow
def test_edge_arrays_past_int32_offsets():
    """270M edges x 8 heads: [E, H] edge arrays hold 2.16e9 elements, so
    their offsets pass 2^31.  Rows of 66,000 edges (split into segments)
    sampled at the start, middle and end of the edge range; the oracle runs
    on the sub-graph of the sampled rows, compared at their positions."""
    n, deg, H, dh = 4096, 66_000, 8, 4
    E = n * deg
    assert E * H > 2**31
    rng = np.random.default_rng(41)
    ind = rng.integers(0, n, size=(n, deg), dtype=np.int32)
    ind.sort(axis=1)
    indptr = (np.arange(n + 1, dtype=np.int64) * deg).astype(np.int32)
    csr = synth.CSR(n, n, indptr, ind.reshape(-1))
    del ind
    G = fg.Graph.from_csr(csr)
    plan = fg.Plan(G, H * dh)
    x = rng.standard_normal((n, H, dh)).astype(np.float32)
    x2 = x.reshape(n, H * dh)
    tx = dev(x)
    rows = np.array([0, 2049, n - 1])
    pos = row_edges(csr, rows)
    sub = synth.CSR(rows.size, n, (np.arange(rows.size + 1) * deg).astype(np.int32),
                    csr.indices[pos])
    tpos = torch.from_numpy(pos).cuda()
    say("edges", E, "sampled rows", rows.tolist(), "last position", int(pos[-1]))
    # SDDMM per head
    s = fg.gsddmm(G, tx, tx, heads=H, plan=plan).reshape(E, H)
    rs, norm = O.gsddmm(sub, x2, x2[rows], heads=H, with_norm=True)
    assert_close_sum(host(s[tpos]), rs.astype(np.float64), norm, dh)
    # edge softmax, the sampled rows given the oracle's scores on both sides
    s[tpos] = dev(rs)
    a = fg.edge_softmax(G, s, leaky=True, slope=0.2, plan=plan).reshape(E, H)
    ra = O.edge_softmax(sub, rs, heads=H, leaky=True, slope=0.2)
    assert_close_softmax(host(a[tpos]), ra, deg)
    del s
    # weighted aggregation with the oracle's weights on the sampled rows
    a[tpos] = dev(ra)
    y = host(fg.gspmm(G, tx, a, msg="src_mul_edge", heads=H, plan=plan)).reshape(n, H * dh)
    ry, rnorm = O.gspmm(sub, x2, msg=O.MSG_SRC_MUL_EDGE, heads=H, edge_val=ra, with_norm=True)
    assert_close_sum(y[rows], ry.astype(np.float64), rnorm, deg)
    del a
    # max with argmax: edge ids near the end of the range
    ym, am = fg.gspmm(G, tx, reduce="max", plan=plan)
    rm, rarg = O.gspmm(sub, x2, red=O.RED_MAX)
    np.testing.assert_array_equal(host(ym).reshape(n, -1)[rows].view(np.uint32), rm.view(np.uint32))
    np.testing.assert_array_equal(host(am).reshape(n, -1)[rows], pos[rarg])


@pytest.mark.slow
def test_features_past_int32_offsets():
    """2.2M vertices x 1,024 features: [N, F] arrays hold 2.25e9 elements, so
    row offsets pass 2^31.  Features come from a seeded torch generator on the
    device; the oracle sees the sampled rows' own sources, relabelled into a
    small sub-graph, and is compared at those rows (sum, max/argmax, SDDMM,
    and the max gradient, fed only at the sampled rows)."""
    n, deg, F = 2_200_000, 4, 1024
    assert n * F > 2**31
    rng = np.random.default_rng(43)
    ind = np.sort(rng.integers(0, n, size=(n, deg), dtype=np.int32), axis=1).reshape(-1)
    indptr = (np.arange(n + 1, dtype=np.int64) * deg).astype(np.int32)
    csr = synth.CSR(n, n, indptr, ind)
    G = fg.Graph.from_csr(csr)
    gen = torch.Generator(device="cuda").manual_seed(44)
    x = torch.randn((n, F), generator=gen, device="cuda")
    rows = np.concatenate([np.arange(n - 40, n), rng.choice(n, 40, replace=False)])
    rows = np.unique(rows).astype(np.int64)
    pos = row_edges(csr, rows)
    uniq, local = np.unique(csr.indices[pos], return_inverse=True)
    sub = synth.CSR(rows.size, uniq.size, (np.arange(rows.size + 1) * deg).astype(np.int32),
                    local.astype(np.int32))
    xs = host(x[torch.from_numpy(uniq.astype(np.int64)).cuda()])
    xd = host(x[torch.from_numpy(rows).cuda()])
    trows = torch.from_numpy(rows).cuda()
    say("rows", n, "features", F, "largest sampled offset", int(rows.max()) * F)
    for plan in (None, fg.Plan(G, F)):
        y = fg.gspmm(G, x, plan=plan)
        ro, norm = O.gspmm(sub, xs, with_norm=True)
        assert_close_sum(host(y[trows]), ro.astype(np.float64), norm, deg)
        del y
        ym, am = fg.gspmm(G, x, reduce="max", plan=plan)
        rm, ra = O.gspmm(sub, xs, red=O.RED_MAX)
        np.testing.assert_array_equal(host(ym[trows]).view(np.uint32), rm.view(np.uint32))
        np.testing.assert_array_equal(host(am[trows]), pos[ra])
        del ym
        sc = fg.gsddmm(G, x, x, plan=plan)
        rs, snorm = O.gsddmm(sub, xs, xd, with_norm=True)
        assert_close_sum(host(sc[torch.from_numpy(pos).cuda()])[:, None], rs.astype(np.float64),
                         snorm, F)
        del sc
        # gradient of max with the upstream gradient nonzero only at the sampled rows
        go = torch.zeros((n, F), device="cuda")
        go_s = np.random.default_rng(45).integers(-4, 5, (rows.size, F)).astype(np.float32)
        go[trows] = dev(go_s)
        gs = fg.gspmm_max_backward(G, am, go, x=x, plan=plan)
        del go, am
        rg = O.gspmm_max_backward(sub, xs, go_s)
        np.testing.assert_array_equal(host(gs[torch.from_numpy(uniq.astype(np.int64)).cuda()]), rg)
        assert float(gs.abs().sum()) == float(np.abs(rg).astype(np.float64).sum())
        del gs


@pytest.mark.slow
def test_rmat_train_step_full():
    w = make_config("rmat_1m_33m_train")
    csr, csc = w.csr, w.csc
    Gf = fg.Graph.from_csr(csr)
    Gb = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
    x, dy = w.arrays["x"], w.arrays["dy"]
    pf, pb = fg.Plan(Gf, 256), fg.Plan(Gb, 256)
    rows_f = sample_rows(csr, 1500, 5)
    rows_b = sample_rows(csc, 1500, 6)
    y = check_spmm(csr, Gf, x, rows=rows_f, plan=pf)
    dx = check_spmm(csc, Gb, dy, rows=rows_b, plan=pb, nnz_total=csr.nnz)
    da = check_sddmm(csr, Gf, x, dy, rows=rows_f, plan=pf)
    # adjoint identity over the whole graph: <dY, A X> = <A^T dY, X> = sum_e dA_e
    tdy, tx = dev(dy).double(), dev(x).double()
    a = float((tdy * y.double()).sum())
    b = float((dx.double() * tx).sum())
    c = float(da.double().sum())
    scale = float((tdy.abs() * fg.gspmm(Gf, dev(np.abs(x)), plan=pf).double()).sum())
    assert abs(a - b) <= 1e-5 * scale and abs(a - c) <= 1e-5 * scale
    # the default plans of this 1 GiB feature matrix use source slabs; the
    # same three without them
    assert pf.info()["num_partitioned_rows"] > 0 and pb.info()["num_partitioned_rows"] > 0
    af, ab = fg.Plan(Gf, 256, source_slab_rows=-2), fg.Plan(Gb, 256, source_slab_rows=-2)
    assert af.info()["num_partitioned_rows"] == 0 and ab.info()["num_partitioned_rows"] == 0
    check_spmm(csr, Gf, x, rows=rows_f, plan=af)
    check_spmm(csc, Gb, dy, rows=rows_b, plan=ab, nnz_total=csr.nnz)
    check_sddmm(csr, Gf, x, dy, rows=rows_f, plan=af)


def test_sddmm_wide_batches_with_edge_ids_and_ragged_ends():
    """The SDDMM's 256-edge batches (items of 128 edges or more on average)
    on a transposed graph with explicit edge ids (ids loaded four per lane,
    scores stored one by one through them) and on its CSR (positional
    16-byte stores): row lengths that are not multiples of 4 or of 256, and
    a stored-edge count that is not a multiple of 4, so the last lane of the
    last item reads its ids one by one.  Also the plain one-edge batches on
    the same graphs (short items), and the sum and max gSpMM on them."""
    rng = np.random.default_rng(77)
    n, m = 700, 900
    deg = rng.integers(150, 420, size=n)
    deg[-1] = 389  # a long last row whose end is not 4-aligned
    dst = np.repeat(np.arange(n), deg)
    src = rng.integers(0, m, size=dst.size)
    assert dst.size % 4 != 0
    csr = synth.coo_to_csr(dst.astype(np.int64), src.astype(np.int64), n, m)
    csc = csr_to_csc(csr)
    for d in (128, 256, 64, 32, 16):
        xs = rng.standard_normal((m, d)).astype(np.float32)
        xd = rng.standard_normal((n, d)).astype(np.float32)
        G = fg.Graph.from_csr(csr)
        for plan in (fg.Plan(G, d), fg.Plan(G, d, segment_edges=64)):
            say("wide-batch SDDMM CSR d=%d items=%d" % (d, plan.info()["num_segments"]))
            check_sddmm(csr, G, xs, xd, plan=plan)
            check_spmm(csr, G, xs, plan=plan)
            check_spmm(csr, G, xs, plan=plan, reduce="max")
        Gt = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
        for plan in (fg.Plan(Gt, d), fg.Plan(Gt, d, segment_edges=64)):
            say("wide-batch SDDMM CSC d=%d items=%d" % (d, plan.info()["num_segments"]))
            check_sddmm(csc, Gt, xd, xs, plan=plan, nnz_total=csr.nnz)


def test_gspmm_wide_batches_ragged_ends():
    """The gSpMM's 256-edge batches (two or more lane groups, long items):
    ids and weights four per lane through the group-major LDS table.  Copy
    and weighted sum, max with and without weights and the MLP's u_add_v
    max, with 2 lane groups at d = 128 (unmasked steps) and d = 100 (every
    step masked), 4 at d = 64, 8 at d = 32 and d = 20 (masked), 16 at
    d = 16, on rows whose lengths are not multiples of 4 or 256 and a
    stored-edge count that is not a multiple of 4 (the last lane of the last
    item loads its ids and weights one by one); then the same graph with
    short items (64-edge batches) and with split rows."""
    rng = np.random.default_rng(78)
    n, m = 600, 1000
    deg = rng.integers(130, 700, size=n)
    deg[5] = 0
    deg[-1] = 517  # a long last row whose end is not 4-aligned
    dst = np.repeat(np.arange(n), deg)
    src = rng.integers(0, m, size=dst.size)
    src[:40] = src[0]  # a run of duplicate edges: ties go to the smallest id
    assert dst.size % 4 != 0
    csr = synth.coo_to_csr(dst.astype(np.int64), src.astype(np.int64), n, m)
    G = fg.Graph.from_csr(csr)
    ew = rng.uniform(0.0, 1.0, csr.nnz).astype(np.float32) + np.float32(1e-3)
    for d in (128, 100, 64, 32, 20, 16):
        x = rng.standard_normal((m, d)).astype(np.float32)
        xi = rng.integers(-4, 5, (m, d)).astype(np.float32)
        ewi = rng.integers(1, 4, csr.nnz).astype(np.float32)
        for plan in (fg.Plan(G, d), fg.Plan(G, d, segment_edges=64),
                     fg.Plan(G, d, segment_edges=300)):
            info = plan.info()
            say("wide-batch gSpMM d=%d items=%d split=%d" % (d, info["num_segments"],
                                                             info["num_split_rows"]))
            check_spmm(csr, G, x, plan=plan)
            check_spmm(csr, G, x, plan=plan, edge=ew)
            check_spmm(csr, G, xi, plan=plan, edge=ewi, exact=True)
            check_spmm(csr, G, x, plan=plan, reduce="max")
            check_spmm(csr, G, xi, plan=plan, reduce="max")
            check_spmm(csr, G, x, plan=plan, edge=ew, reduce="max")
    xm = rng.standard_normal((m, 8)).astype(np.float32)
    xdm = rng.standard_normal((n, 8)).astype(np.float32)
    for d_out in (128, 32, 16):
        w = rng.standard_normal((8, d_out)).astype(np.float32)
        for plan in (fg.Plan(G, d_out), fg.Plan(G, d_out, segment_edges=300)):
            check_mlp(csr, G, xm, xdm, w, plan=plan)


def test_wide_batches_for_many_lane_groups_on_mid_length_rows():
    """Items of 64 to 127 edges on average: kernels with four or more lane
    groups (d <= 64) take the wide batches, two groups (d = 128) keep 64-edge
    batches.  Rows of 60-130 edges (one or two 64-edge batches, never more
    than one wide batch), an empty row and a last row that ends off a
    4-edge boundary."""
    rng = np.random.default_rng(80)
    n, m = 900, 700
    deg = rng.integers(60, 131, size=n)
    deg[11] = 0
    deg[-1] = 83
    dst = np.repeat(np.arange(n), deg)
    src = rng.integers(0, m, size=dst.size)
    if dst.size % 4 == 0:
        dst, src = dst[:-1], src[:-1]
    csr = synth.coo_to_csr(dst.astype(np.int64), src.astype(np.int64), n, m)
    G = fg.Graph.from_csr(csr)
    ew = rng.uniform(0.0, 1.0, csr.nnz).astype(np.float32) + np.float32(1e-3)
    for d in (16, 32, 48, 64, 128):
        xs = rng.standard_normal((m, d)).astype(np.float32)
        xd = rng.standard_normal((n, d)).astype(np.float32)
        plan = fg.Plan(G, d)
        say("mid-length rows d=%d items=%d" % (d, plan.info()["num_segments"]))
        for pl in (plan, None):
            check_spmm(csr, G, xs, plan=pl)
            check_spmm(csr, G, xs, plan=pl, edge=ew)
            check_spmm(csr, G, xs, plan=pl, reduce="max")
            check_sddmm(csr, G, xs, xd, plan=pl)


def test_gat_fused_wide_batches_ragged_ends():
    """The fused attention kernel's 256-edge batches (two lane groups, F = 128,
    items of 128 edges or more on average) with ids through the group-major
    LDS table: heads of 16, 64 and 128 features, rows whose lengths are not
    multiples of 4 or 256, a stored-edge count that is not a multiple of 4,
    an empty row; whole rows and split rows."""
    rng = np.random.default_rng(79)
    n = 800
    deg = rng.integers(130, 600, size=n)
    deg[7] = 0
    deg[-1] = 301
    dst = np.repeat(np.arange(n), deg)
    src = rng.integers(0, n, size=dst.size)
    assert dst.size % 4 != 0
    csr = synth.coo_to_csr(dst.astype(np.int64), src.astype(np.int64), n, n)
    G = fg.Graph.from_csr(csr)
    for heads, dh in ((8, 16), (2, 64), (1, 128)):
        x = (rng.standard_normal((n, heads, dh)) * 0.25).astype(np.float32)
        for plan in (fg.Plan(G, heads * dh), fg.Plan(G, heads * dh, segment_edges=1000)):
            info = plan.info()
            say("wide-batch attention H=%d dh=%d items=%d split=%d" % (
                heads, dh, info["num_segments"], info["num_split_rows"]))
            check_gat(csr, G, x, plan=plan, heads=heads)


def test_sddmm_own_schedule_on_spread_graph():
    """A spread graph with source slabs at d >= 256: the plan holds a schedule
    of its own for the SDDMM (every row cut at slab boundaries, no slots),
    which fg_gsddmm runs; checked on every row, on the CSR and on the CSC
    with explicit edge ids, and the gSpMM of the same plan alongside."""
    rng = np.random.default_rng(9)
    n, m, deg = 3000, 30000, 100
    dst = np.repeat(np.arange(n), deg)
    src = rng.integers(0, m, size=n * deg)
    csr = synth.coo_to_csr(dst.astype(np.int64), src.astype(np.int64), n, m)
    csc = csr_to_csc(csr)
    for d in (256, 512):
        xs = rng.standard_normal((m, d)).astype(np.float32)
        xd = rng.standard_normal((n, d)).astype(np.float32)
        G = fg.Graph.from_csr(csr)
        plan = fg.Plan(G, d, source_slab_rows=4096)
        info = plan.info()
        say("SDDMM schedule d=%d: %d items (gather %d)" % (d, info["sddmm_segments"],
                                                          info["num_segments"]))
        assert info["sddmm_segments"] > info["num_segments"]
        check_sddmm(csr, G, xs, xd, plan=plan)
        check_spmm(csr, G, xs, plan=plan)
        Gt = fg.Graph.from_csr(csc, nnz_total=csr.nnz)
        pt = fg.Plan(Gt, d, source_slab_rows=4096)
        check_sddmm(csc, Gt, xd, xs, plan=pt, nnz_total=csr.nnz)
