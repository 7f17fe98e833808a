"""C-ABI checks that need no GPU: the library loads, exports every symbol the
public header declares, rejects invalid arguments on the host before any
launch, and builds a correct degree-aware schedule."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest
import torch

import paper_2008_11359_amd as fg
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "featgraph_hip.h")


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fg_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared_functions()
    assert len(names) >= 9
    out = subprocess.run(["nm", "-D", "--defined-only", fg.LIB_PATH], check=True,
                         capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (fg_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    for n in names:
        getattr(fg._lib, n)  # resolvable through ctypes too


def test_version_and_status_strings():
    assert fg._lib.fg_abi_version() == fg.ABI_VERSION == 4
    for s in (0, -1, -2, -3, -4, -5):
        assert fg.status_string(s) and fg.status_string(s) != "unknown status"
    assert fg.status_string(7) == "unknown status"


def _graph_struct(num_rows=4, num_cols=4, nnz=7, nnz_total=0, fake=0x1000):
    # fake, never dereferenced: every call below must fail host validation first
    return fg._Graph(num_rows, num_cols, nnz, nnz_total, fake, fake + 0x100, None)


FAKE_X, FAKE_OUT, FAKE_ARG, FAKE_EV = 0x10000, 0x20000, 0x30000, 0x40000


@pytest.mark.parametrize("case", [
    "null_graph", "neg_rows", "huge_nnz", "no_indptr", "zero_heads", "zero_dh", "too_wide",
    "bad_msg", "bad_red", "mul_without_edge", "copy_with_edge", "max_without_arg",
    "sum_with_arg", "no_x", "no_out", "out_aliases_x", "nnz_total_too_small"])
@pytest.mark.parametrize("entry", ["fg_gspmm", "fg_gspmm_noalloc"])
def test_gspmm_rejects_invalid_arguments(case, entry):
    """Both gSpMM entry points share their host checks; the allocation-free
    one must reject before it touches the device (there is none here)."""
    L = fg._lib
    g = _graph_struct()
    args = dict(msg=0, red=0, H=1, dh=4, x=FAKE_X, ev=None, out=FAKE_OUT, arg=None)
    gp = ctypes.byref(g)
    if case == "null_graph":
        gp = None
    elif case == "neg_rows":
        g.num_rows = -1
    elif case == "huge_nnz":
        g.nnz = 1 << 31
    elif case == "no_indptr":
        g.indptr = None
    elif case == "zero_heads":
        args["H"] = 0
    elif case == "zero_dh":
        args["dh"] = 0
    elif case == "too_wide":
        args["H"], args["dh"] = 1 << 9, 1 << 8
    elif case == "bad_msg":
        args["msg"] = 5
    elif case == "bad_red":
        args["red"] = -1
    elif case == "mul_without_edge":
        args["msg"] = 1
    elif case == "copy_with_edge":
        args["ev"] = FAKE_EV
    elif case == "max_without_arg":
        args["red"] = 1
    elif case == "sum_with_arg":
        args["arg"] = FAKE_ARG
    elif case == "no_x":
        args["x"] = None
    elif case == "no_out":
        args["out"] = None
    elif case == "out_aliases_x":
        args["out"] = FAKE_X + 8
    elif case == "nnz_total_too_small":
        g.nnz_total = 3
    st = getattr(L, entry)(gp, args["msg"], args["red"], args["H"], args["dh"], args["x"],
                           args["ev"], args["out"], args["arg"], None, None)
    assert st == fg.FG_ERR_INVALID_ARG


@pytest.mark.parametrize("case", ["bad_op", "no_xs", "no_out", "out_aliases_xd", "bad_heads"])
def test_gsddmm_rejects_invalid_arguments(case):
    L = fg._lib
    g = _graph_struct()
    op, H, dh, xs, xd, out = 0, 1, 4, FAKE_X, FAKE_X + 0x1000, FAKE_OUT
    if case == "bad_op":
        op = 3
    elif case == "no_xs":
        xs = None
    elif case == "no_out":
        out = None
    elif case == "out_aliases_xd":
        out = xd + 4
    elif case == "bad_heads":
        H = -2
    assert L.fg_gsddmm(ctypes.byref(g), op, H, dh, xs, xd, out, None, None) == fg.FG_ERR_INVALID_ARG


def test_edge_softmax_rejects_invalid_arguments():
    L = fg._lib
    g = _graph_struct()
    assert L.fg_edge_softmax(ctypes.byref(g), 0, FAKE_X, 1, 0.2, FAKE_OUT, None, None) == -1
    assert L.fg_edge_softmax(ctypes.byref(g), 1, None, 1, 0.2, FAKE_OUT, None, None) == -1
    # partial overlap of out and scores (exact aliasing is allowed)
    assert L.fg_edge_softmax(ctypes.byref(g), 1, FAKE_X, 1, 0.2, FAKE_X + 4, None, None) == -1


def test_gsddmm_edge_softmax_rejects_invalid_arguments():
    L = fg._lib
    g = _graph_struct()
    XS, XD, SC, OUT = 0x10000, 0x20000, 0x30000, 0x40000

    def call(H=1, dh=8, xs=XS, xd=XD, sc=SC, out=OUT):
        return L.fg_gsddmm_edge_softmax(ctypes.byref(g), H, dh, xs, xd, 1, 0.2, sc, out, None,
                                        None)

    assert call(H=0) == fg.FG_ERR_INVALID_ARG
    assert call(dh=0) == fg.FG_ERR_INVALID_ARG
    assert call(xs=None) == fg.FG_ERR_INVALID_ARG
    assert call(sc=None) == fg.FG_ERR_INVALID_ARG
    assert call(out=None) == fg.FG_ERR_INVALID_ARG
    assert call(out=SC + 4) == fg.FG_ERR_INVALID_ARG   # weights overlap the scores
    assert call(sc=XS + 16) == fg.FG_ERR_INVALID_ARG   # scores overlap x_src


def test_gat_aggregate_rejects_invalid_or_unsupported_arguments():
    L = fg._lib
    g = _graph_struct()
    ok = dict(H=2, dh=8, xs=FAKE_X, xd=FAKE_X + 0x1000, out=FAKE_OUT)

    def call(**kw):
        a = dict(ok, **kw)
        return L.fg_gat_aggregate(ctypes.byref(g), a["H"], a["dh"], a["xs"], a["xd"], 1, 0.2,
                                  a["out"], None, None)

    assert call(H=0) == fg.FG_ERR_INVALID_ARG
    assert call(xs=None) == fg.FG_ERR_INVALID_ARG
    assert call(out=None) == fg.FG_ERR_INVALID_ARG
    assert call(out=FAKE_X + 16) == fg.FG_ERR_INVALID_ARG  # overlaps x_src
    # valid but outside the fused kernel's shapes
    assert call(dh=6) == fg.FG_ERR_UNSUPPORTED     # dh not a multiple of 4
    assert call(dh=12) == fg.FG_ERR_UNSUPPORTED    # 3 lanes per head
    assert call(H=8, dh=64) == fg.FG_ERR_UNSUPPORTED  # wider than 256
    assert call(xs=FAKE_X + 4) == fg.FG_ERR_UNSUPPORTED  # not 16-byte aligned


def test_gspmm_max_backward_rejects_invalid_arguments():
    L = fg._lib
    g = _graph_struct()
    GS, GE, GO = 0x50000, 0x60000, 0x70000
    ok = dict(msg=0, H=1, dh=4, x=FAKE_X, ev=None, arg=FAKE_ARG, go=GO, gs=GS, ge=None)

    def call(graph=g, **kw):
        a = dict(ok, **kw)
        return L.fg_gspmm_max_backward(ctypes.byref(graph), a["msg"], a["H"], a["dh"], a["x"],
                                       a["ev"], a["arg"], a["go"], a["gs"], a["ge"], None, None)

    assert call(msg=2) == fg.FG_ERR_INVALID_ARG
    assert call(H=0) == fg.FG_ERR_INVALID_ARG
    assert call(ev=FAKE_EV) == fg.FG_ERR_INVALID_ARG           # copy_src takes no edge values
    assert call(ge=GE) == fg.FG_ERR_INVALID_ARG                # ... and has no edge gradient
    assert call(msg=1) == fg.FG_ERR_INVALID_ARG                # src_mul_edge without values
    assert call(msg=1, ev=FAKE_EV, ge=GE, x=None) == fg.FG_ERR_INVALID_ARG  # edge grad needs x
    assert call(arg=None) == fg.FG_ERR_INVALID_ARG
    assert call(go=None) == fg.FG_ERR_INVALID_ARG
    assert call(gs=FAKE_X + 4) == fg.FG_ERR_INVALID_ARG        # output overlaps x
    assert call(gs=GO + 8) == fg.FG_ERR_INVALID_ARG            # output overlaps grad_out
    assert call(msg=1, ev=FAKE_EV, ge=GS + 4) == fg.FG_ERR_INVALID_ARG  # the two outputs overlap
    eg = fg._Graph(4, 4, 7, 7, 0x1000, 0x1100, 0x1200)
    assert call(graph=eg) == fg.FG_ERR_INVALID_ARG             # edge ids need the graph's plan


def test_edge_softmax_backward_rejects_invalid_arguments():
    L = fg._lib
    g = _graph_struct()
    A, GO, S, DS = 0x10000, 0x20000, 0x30000, 0x40000

    def call(H=1, a=A, go=GO, s=S, leaky=1, ds=DS):
        return L.fg_edge_softmax_backward(ctypes.byref(g), H, a, go, s, leaky, 0.2, ds, None, None)

    assert call(H=0) == fg.FG_ERR_INVALID_ARG
    assert call(a=None) == fg.FG_ERR_INVALID_ARG
    assert call(go=None) == fg.FG_ERR_INVALID_ARG
    assert call(ds=None) == fg.FG_ERR_INVALID_ARG
    assert call(s=None) == fg.FG_ERR_INVALID_ARG               # leaky needs the scores
    assert call(ds=A + 4) == fg.FG_ERR_INVALID_ARG             # overlaps the weights
    assert call(ds=S) == fg.FG_ERR_INVALID_ARG                 # overlaps the scores
    assert call(ds=GO + 4) == fg.FG_ERR_INVALID_ARG            # partial overlap of grad_out


def test_gsddmm_edge_softmax_backward_rejects_invalid_arguments():
    L = fg._lib
    g = _graph_struct()  # 4 x 4, 7 edges
    XS, XD, A, S, DS = 0x10000, 0x20000, 0x30000, 0x40000, 0x50000

    def call(H=2, dh=16, xs=XS, xd=XD, a=A, s=S, leaky=1, ds=DS):
        return L.fg_gsddmm_edge_softmax_backward(ctypes.byref(g), H, dh, xs, xd, a, s, leaky, 0.2,
                                                 ds, None, None)

    assert call(H=0) == fg.FG_ERR_INVALID_ARG
    assert call(dh=0) == fg.FG_ERR_INVALID_ARG
    for k in ("xs", "xd", "a", "ds"):
        assert call(**{k: None}) == fg.FG_ERR_INVALID_ARG
    assert call(s=None) == fg.FG_ERR_INVALID_ARG               # leaky needs the scores
    assert call(ds=A + 4) == fg.FG_ERR_INVALID_ARG             # overlaps the weights
    assert call(ds=S) == fg.FG_ERR_INVALID_ARG                 # overlaps the scores
    assert call(ds=XS + 8) == fg.FG_ERR_INVALID_ARG            # overlaps the source features
    assert call(ds=XD) == fg.FG_ERR_INVALID_ARG                # overlaps the destination features


def test_dense_matmul_rejects_invalid_arguments():
    L = fg._lib
    X, W, Y = 0x10000, 0x20000, 0x30000
    assert L.fg_dense_matmul(-1, 8, 8, X, W, Y, None) == fg.FG_ERR_INVALID_ARG
    assert L.fg_dense_matmul(4, 0, 8, X, W, Y, None) == fg.FG_ERR_INVALID_ARG
    assert L.fg_dense_matmul(4, 8, 1 << 17, X, W, Y, None) == fg.FG_ERR_INVALID_ARG
    assert L.fg_dense_matmul(4, 8, 8, None, W, Y, None) == fg.FG_ERR_INVALID_ARG
    assert L.fg_dense_matmul(4, 8, 8, X, W, X + 16, None) == fg.FG_ERR_INVALID_ARG  # y overlaps x
    assert L.fg_dense_matmul(0, 8, 8, None, None, None, None) == fg.FG_OK  # nothing to do


def test_mlp_aggregate_rejects_invalid_arguments():
    L = fg._lib
    g = _graph_struct()
    XS, XD, W, OUT, ARG, WS = 0x10000, 0x20000, 0x30000, 0x40000, 0x50000, 0x60000
    ok = dict(di=8, do=16, xs=XS, xd=XD, w=W, out=OUT, arg=ARG, ws=WS)

    def call(**kw):
        a = dict(ok, **kw)
        return L.fg_mlp_aggregate(ctypes.byref(g), a["di"], a["do"], a["xs"], a["xd"], a["w"],
                                  a["out"], a["arg"], a["ws"], None, None)

    assert call(di=0) == fg.FG_ERR_INVALID_ARG
    assert call(do=0) == fg.FG_ERR_INVALID_ARG
    assert call(xs=None) == fg.FG_ERR_INVALID_ARG
    assert call(w=None) == fg.FG_ERR_INVALID_ARG
    assert call(arg=None) == fg.FG_ERR_INVALID_ARG
    assert call(ws=None) == fg.FG_ERR_INVALID_ARG
    assert call(out=XS + 8) == fg.FG_ERR_INVALID_ARG   # overlaps x_src
    assert call(ws=OUT + 4) == fg.FG_ERR_INVALID_ARG   # workspace overlaps out
    g2 = _graph_struct(num_rows=4, num_cols=5)
    assert L.fg_mlp_aggregate(ctypes.byref(g2), 8, 16, XS, XS, W, OUT, ARG, WS, None, None) == \
        fg.FG_ERR_INVALID_ARG  # x_dst = x_src needs a square graph


def test_plan_create_rejects_invalid_arguments():
    L = fg._lib
    g = _graph_struct()
    h = ctypes.c_void_p()
    opt = fg._PlanOptions()
    assert L.fg_plan_create(ctypes.byref(g), None, None, 0, None, ctypes.byref(h), None) == -1
    assert L.fg_plan_create(ctypes.byref(g), None, None, 8, None, None, None) == -1
    opt.reserved[0] = 1
    assert L.fg_plan_create(ctypes.byref(g), None, None, 8, ctypes.byref(opt), ctypes.byref(h),
                            None) == -1
    opt.reserved[0] = 0
    opt.max_backward = 2  # 0 or 1
    assert L.fg_plan_create(ctypes.byref(g), None, None, 8, ctypes.byref(opt), ctypes.byref(h),
                            None) == -1
    # the binned max-backward records need rows x max_width <= 2^31 - 1 (int32
    # offsets): refused before any device work
    opt.max_backward = 1
    big = _graph_struct(num_rows=1 << 20, num_cols=8, nnz=7)
    assert L.fg_plan_create(ctypes.byref(big), None, None, 4096, ctypes.byref(opt),
                            ctypes.byref(h), None) == fg.FG_ERR_UNSUPPORTED
    assert not h.value
    opt.max_backward = 0
    opt.max_row_segments = 1  # a row must be allowed at least two pieces
    assert L.fg_plan_create(ctypes.byref(g), None, None, 8, ctypes.byref(opt), ctypes.byref(h),
                            None) == -1
    opt.max_row_segments = 0
    opt.segment_edges = -5
    assert L.fg_plan_create(ctypes.byref(g), None, None, 8, ctypes.byref(opt), ctypes.byref(h),
                            None) == -1
    opt.segment_edges = 0
    opt.partition_min_degree = -1
    assert L.fg_plan_create(ctypes.byref(g), None, None, 8, ctypes.byref(opt), ctypes.byref(h),
                            None) == -1
    # an inconsistent host indptr is rejected before any device allocation
    ip = np.array([0, 3, 2, 4, 7], np.int32)
    assert L.fg_plan_create(ctypes.byref(g), ip.ctypes.data, None, 8, None, ctypes.byref(h),
                            None) == -1
    ip = np.array([0, 3, 4, 4, 6], np.int32)  # last entry != nnz
    assert L.fg_plan_create(ctypes.byref(g), ip.ctypes.data, None, 8, None, ctypes.byref(h),
                            None) == -1
    ip = np.array([0, 3, 4, 4, 7], np.int32)
    ix = np.array([0, 1, 2, 3, 0, 4, 1], np.int32)  # source 4 >= num_cols
    assert L.fg_plan_create(ctypes.byref(g), ip.ctypes.data, ix.ctypes.data, 8, None,
                            ctypes.byref(h), None) == -1
    assert L.fg_plan_destroy(None) == -1
    assert L.fg_plan_get_info(None, None) == -1


def test_binding_refuses_cpu_tensors():
    csr = synth.small_random_graph(np.random.default_rng(0), 8, 8, 20)
    with pytest.raises((ValueError, RuntimeError, AssertionError)):
        fg.Graph(8, 8, torch.from_numpy(csr.indptr), torch.from_numpy(csr.indices))


# ---------------------------------------------------------------- schedule


def _check_schedule(indptr, S, cap=128, indices=None, num_cols=0, slab=0, min_deg=0,
                    which="plain", max_width=128):
    segs, n_split, n_slot = fg.schedule_host(
        indptr, indices, num_cols, max_width, which, segment_edges=S, max_row_segments=cap,
        source_slab_rows=slab, partition_min_degree=min_deg)
    num_rows = indptr.size - 1
    deg = np.diff(indptr.astype(np.int64))
    pad = segs[:, 0] < 0
    assert np.all(segs[pad, 1:] == [0, 0, -1])  # padding items are empty
    real = segs[~pad]
    # every edge covered exactly once, every row present
    cover = np.zeros(int(indptr[-1]), np.int32)
    pieces = np.zeros(num_rows, np.int64)
    for r, b, e, sl in real:
        assert indptr[r] <= b <= e <= indptr[r + 1]
        cover[b:e] += 1
        pieces[r] += 1
    assert np.all(cover == 1)
    assert np.all(pieces >= 1)
    # slots: rows with several pieces, numbered consecutively per row in edge order
    split = pieces >= 2
    assert n_split == int(split.sum())
    assert n_slot == int(pieces[split].sum())
    slotted = real[real[:, 3] >= 0]
    assert np.array_equal(np.sort(slotted[:, 3]), np.arange(n_slot))
    assert np.all(split[slotted[:, 0]]) and np.all(~split[real[real[:, 3] < 0, 0]])
    by_slot = slotted[np.argsort(slotted[:, 3])]
    for r in np.nonzero(split)[0][:200]:
        rs = by_slot[by_slot[:, 0] == r]
        assert np.all(np.diff(rs[:, 3]) == 1)
        assert rs[0, 1] == indptr[r] and rs[-1, 2] == indptr[r + 1]
        assert np.all(rs[1:, 1] == rs[:-1, 2])  # slot order = edge order
    lens = real[:, 2] - real[:, 1]
    if which == "plain" or indices is None:
        k = np.minimum(np.maximum(-(-deg // S), 1), cap)
        assert np.array_equal(pieces, k)
        assert np.all(lens <= np.maximum(S, -(-deg[real[:, 0]] // cap)))
        assert not pad.any()
        # longest first (rows without edges last), or by power-of-two length
        # class (ceil(log2(len))) with rows in id order within a class;
        # without indices always the former
        cls = np.where(lens > 0, np.ceil(np.log2(np.maximum(lens, 1))), -1).astype(np.int64)
        assert np.all(np.diff(cls) <= 0)
        by_len = bool(np.all(np.diff(lens) <= 0))
        by_id = bool(np.all(np.diff(real[:, 0])[np.diff(cls) == 0] >= 0))
        assert by_len or by_id
        assert by_len or indices is not None
        return segs
    # gather schedule with source slabs
    nslab = -(-num_cols // slab)
    thresh = min_deg if min_deg else max(64, 8 * nslab)
    part = deg >= thresh
    for r in np.nonzero(part)[0]:
        row = indices[indptr[r]:indptr[r + 1]]
        part[r] = bool(np.all(np.diff(row) >= 0))
    is_part = part[real[:, 0]]
    lo = indices[real[is_part, 1]].astype(np.int64)       # smallest source of a piece
    hi = indices[real[is_part, 2] - 1].astype(np.int64)   # largest source of a piece
    assert np.all(hi - lo < slab)  # a piece lies inside one slab of at most `slab` ids
    assert np.all(lens[is_part] <= S)
    # stream of die x = workgroups (4 items) w with w % 8 == x
    die = ((np.nonzero(~pad)[0] // 4) % 8)[is_part]
    for x in range(8):  # each die walks its slabs in source order
        assert np.all(np.diff(lo[die == x]) >= -(slab - 1))
        assert np.all(np.diff(hi[die == x]) >= -(slab - 1))
    # pieces on different dies come from disjoint source ranges (a slab, and
    # with it its feature rows, belongs to one die)
    order = np.argsort(lo, kind="stable")
    lo_s, hi_s, die_s = lo[order], hi[order], die[order]
    run_hi = np.maximum.accumulate(hi_s)
    cross = die_s[1:] != die_s[:-1]
    assert np.all(lo_s[1:][cross] > run_hi[:-1][cross])
    return segs


@pytest.mark.parametrize("S,cap", [(1, 128), (7, 128), (64, 2), (64, 128), (1024, 4)])
def test_schedule_covers_every_edge(S, cap):
    w = synth.make_config("rmat_233k_115m", scale_down=512)
    _check_schedule(w.csr.indptr, S, cap)


@pytest.mark.parametrize("S,slab,min_deg", [(4096, 64, 0), (64, 16, 8), (7, 100, 1)])
def test_partitioned_schedule(S, slab, min_deg):
    w = synth.make_config("rmat_233k_115m", scale_down=128)
    c = w.csr
    segs = _check_schedule(c.indptr, S, indices=c.indices, num_cols=c.num_cols, slab=slab,
                           min_deg=min_deg, which="gather")
    assert (segs[:, 0] >= 0).sum() > c.num_rows  # some rows were cut
    # the plain schedule of the same graph ignores the slabs
    _check_schedule(c.indptr, S, indices=c.indices, num_cols=c.num_cols, slab=slab,
                    min_deg=min_deg, which="plain")


def test_partition_min_degree_default_and_explicit():
    """Rows of 100 edges over 16 id slabs: the default minimum (8 edges a
    piece, 128) leaves them whole; an explicit minimum of 64 cuts them."""
    w = synth.make_config("uniform_deg100_100k", d=8, scale_down=50)
    c = w.csr
    slab = -(-c.num_cols // 16)
    segs, _, n_slot = fg.schedule_host(c.indptr, c.indices, c.num_cols, 128, "gather",
                                       source_slab_rows=slab)
    assert n_slot == 0
    segs = _check_schedule(c.indptr, 4096, indices=c.indices, num_cols=c.num_cols, slab=slab,
                           min_deg=64, which="gather")
    assert (segs[:, 0] >= 0).sum() >= 12 * c.num_rows


def test_partition_automatic_slabs():
    """source_slab_rows < 0 picks slabs of max(8 MiB of features, num_cols /
    16) ids and the default minimum row length for that many slabs."""
    w = synth.make_config("uniform_deg100_100k", d=8, scale_down=5)
    c = w.csr
    # 20,000 sources x 256 floats = 20 MB: fits the dies' L2s, no partitioning
    auto = fg.schedule_host(c.indptr, c.indices, c.num_cols, 256, "gather", source_slab_rows=-1)
    assert auto[2] == 0 and auto[0].shape[0] == c.num_rows
    for width in (512, 1024, 4096):
        slab = max(64, (8 << 20) // (4 * width), -(-c.num_cols // 16))
        auto = fg.schedule_host(c.indptr, c.indices, c.num_cols, width, "gather",
                                source_slab_rows=-1)
        same = fg.schedule_host(c.indptr, c.indices, c.num_cols, width, "gather",
                                source_slab_rows=slab)
        np.testing.assert_array_equal(auto[0], same[0])
        nslab = -(-c.num_cols // slab)
        segs = _check_schedule(c.indptr, 4096, indices=c.indices, num_cols=c.num_cols,
                               slab=slab, which="gather")
        if max(64, 8 * nslab) <= 100:  # rows of 100 edges are cut
            assert (segs[:, 0] >= 0).sum() >= 7 * c.num_rows and auto[2] > 0
        else:
            assert (segs[:, 0] >= 0).sum() == c.num_rows and auto[2] == 0


def test_partition_default_rule():
    """By default the gather schedule uses automatic slabs once the num_cols x
    max_width features exceed 128 MiB, or 32 MiB when the gathers are spread
    (the most used 4 MB of source rows take under 45% of the edges and rows
    with neighbouring ids do not share sources); -2 switches slabs off, below
    -2 is an error."""
    w = synth.make_config("rand_100k_48m", d=16, scale_down=5)  # 20,000 ids, hot rows ~2000 edges
    c = w.csr
    plain = {wd: fg.schedule_host(c.indptr, None, c.num_cols, wd, "gather") for wd in (256, 1024, 4096)}
    # 20,000 x 256 floats = 20 MB: no slabs
    np.testing.assert_array_equal(
        fg.schedule_host(c.indptr, c.indices, c.num_cols, 256, "gather")[0], plain[256][0])
    # 82 MB and spread (the top 1,024 sources take 22% of the edges): slabs
    spread = fg.schedule_host(c.indptr, c.indices, c.num_cols, 1024, "gather")
    np.testing.assert_array_equal(
        spread[0], fg.schedule_host(c.indptr, c.indices, c.num_cols, 1024, "gather",
                                    source_slab_rows=-1)[0])
    assert spread[0].shape[0] > plain[1024][0].shape[0]
    # 328 MB: the automatic slabs of source_slab_rows=-1, unconditionally
    above = fg.schedule_host(c.indptr, c.indices, c.num_cols, 4096, "gather")
    auto = fg.schedule_host(c.indptr, c.indices, c.num_cols, 4096, "gather", source_slab_rows=-1)
    np.testing.assert_array_equal(above[0], auto[0])
    assert above[0].shape[0] > plain[4096][0].shape[0]
    off = fg.schedule_host(c.indptr, c.indices, c.num_cols, 4096, "gather", source_slab_rows=-2)
    np.testing.assert_array_equal(off[0], plain[4096][0])
    with pytest.raises(fg.FgError):
        fg.schedule_host(c.indptr, c.indices, c.num_cols, 4096, "gather", source_slab_rows=-3)


@pytest.mark.parametrize("name,cut", [
    ("rmat_233k_115m", False),        # hubs: the top 1,024 sources take 60% of the edges
    ("clustered_133k_deg300", False),  # spread, but neighbouring ids share sources
    ("uniform_deg100_100k", True),     # spread: 6%
])
def test_partition_spread_gathers(name, cut):
    """Between 32 and 128 MiB of features (width 1,024 on a tenth- or
    fifth-size graph), slabs only for spread gathers without id locality."""
    sd = 5 if name == "uniform_deg100_100k" else 10
    w = synth.make_config(name, d=16 if name == "uniform_deg100_100k" else None, scale_down=sd)
    c = w.csr
    assert 32 << 20 < c.num_cols * 1024 * 4 <= 128 << 20
    d = fg.schedule_host(c.indptr, c.indices, c.num_cols, 1024, "gather")
    plain = fg.schedule_host(c.indptr, None, c.num_cols, 1024, "gather")
    assert (d[0].shape[0] != plain[0].shape[0] or d[2] != plain[2]) == cut


def test_partition_slabs_balance_dies():
    """Busy sources labelled first (one id slab would hold most edges): the
    slabs follow the edges, so the partitioned work spreads over all dies."""
    w = synth.make_config("rand_100k_48m", d=16, scale_down=20)
    g = w.csr
    outdeg = np.bincount(g.indices, minlength=g.num_cols)
    order = np.argsort(-outdeg, kind="stable")
    rank = np.empty_like(order)
    rank[order] = np.arange(order.size)
    hf = synth.coo_to_csr(rank[synth.csr_rows(g)], rank[g.indices], g.num_rows, g.num_cols)
    segs = _check_schedule(hf.indptr, 4096, indices=hf.indices, num_cols=hf.num_cols,
                           slab=1024, min_deg=500, which="gather")
    real = segs[segs[:, 0] >= 0]
    big = np.diff(hf.indptr.astype(np.int64))[real[:, 0]] >= 500
    die = ((np.nonzero(segs[:, 0] >= 0)[0] // 4) % 8)[big]
    per_die = np.bincount(die, weights=(real[big, 2] - real[big, 1]), minlength=8)
    assert per_die.min() > 0.8 * per_die.mean()


def test_schedule_with_indices_but_no_slabs():
    """Indices without source partitioning give the plain cut."""
    w = synth.make_config("rmat_233k_115m", scale_down=512)
    c = w.csr
    a = fg.schedule_host(c.indptr, c.indices, c.num_cols, 128, "gather", segment_edges=64)
    b = fg.schedule_host(c.indptr, None, c.num_cols, 128, "gather", segment_edges=64)
    np.testing.assert_array_equal(a[0], b[0])
    assert a[1:] == b[1:]


def test_partitioning_skips_unsorted_rows():
    ip = np.array([0, 300, 300], np.int32)
    ix = np.random.default_rng(0).integers(0, 1000, 300).astype(np.int32)  # unsorted hub
    segs, n_split, n_slot = fg.schedule_host(ip, ix, 1000, 128, "gather", segment_edges=64,
                                             source_slab_rows=250, partition_min_degree=1)
    assert n_slot == 5 and not (segs[:, 0] < 0).any()  # plain cut: ceil(300 / 64)
    ix.sort()
    segs, n_split, n_slot = fg.schedule_host(ip, ix, 1000, 128, "gather", segment_edges=64,
                                             source_slab_rows=250, partition_min_degree=1)
    assert n_slot > 5  # now cut at slab boundaries too


def test_schedule_edge_cases():
    _check_schedule(np.zeros(1, np.int32), 8)            # no rows
    _check_schedule(np.zeros(6, np.int32), 8)            # only empty rows
    _check_schedule(np.array([0, 100], np.int32), 8)     # one hub row
    _check_schedule(np.array([0, 8, 16, 17], np.int32), 8)
    with pytest.raises(fg.FgError):
        fg.schedule_host(np.array([0, 5, 3], np.int32), segment_edges=8)
    with pytest.raises(fg.FgError):  # a source id out of range
        fg.schedule_host(np.array([0, 2], np.int32), np.array([0, 9], np.int32), 5)


def _fnv1a64(ip):
    h = 14695981039346656037
    for b in np.ascontiguousarray(ip, dtype="<i4").tobytes():
        h = ((h ^ b) * 1099511628211) & 0xFFFFFFFFFFFFFFFF
    return h


def test_indptr_checksum_is_fnv1a_and_sees_in_place_edits():
    ip = np.array([0, 3, 4, 4, 7], np.int32)
    assert fg.indptr_checksum(ip) == _fnv1a64(ip)
    moved = ip.copy()
    moved[1] = 2  # one edge moved from row 0 to row 1: same shape and nnz
    assert fg.indptr_checksum(moved) != fg.indptr_checksum(ip)
    big = synth.make_config("tiny_uniform_1k").csr.indptr
    assert fg.indptr_checksum(big) == _fnv1a64(big)
    out = ctypes.c_uint64()
    assert fg._lib.fg_indptr_checksum(None, 4, ctypes.byref(out)) == fg.FG_ERR_INVALID_ARG
    assert fg._lib.fg_indptr_checksum(ip.ctypes.data, -1, ctypes.byref(out)) == \
        fg.FG_ERR_INVALID_ARG
    assert fg._lib.fg_plan_validate(None, None, None, None) == fg.FG_ERR_INVALID_ARG


def test_plan_refuses_a_graph_edited_in_place():
    """The binding records the in-place modification counters of the graph's
    arrays when a plan is built and refuses the plan once any of them moved
    (the kernels take row ranges from the plan, not from indptr)."""
    from types import SimpleNamespace

    p = fg.Plan.__new__(fg.Plan)
    p._h = None
    p.graph = SimpleNamespace(indptr=torch.tensor([0, 3, 4, 4, 7], dtype=torch.int32),
                              indices=torch.zeros(7, dtype=torch.int32), edge_ids=None)
    p._versions = fg._graph_versions(p.graph)
    p.check_current()
    p.graph.indices[2] = 1
    with pytest.raises(ValueError, match="modified in place"):
        p.check_current()
    p._versions = fg._graph_versions(p.graph)
    p.graph.indptr[1] = 2
    with pytest.raises(ValueError, match="modified in place"):
        fg._plan_handle(p)


@pytest.mark.parametrize("S", [64, 4096])
def test_die_banded_schedule(S):
    """item_order 3 with band_row_edges = -1: the gather schedule holds the
    plain schedule's items (same pieces, same slots), piece k of a row cut into K >= 8 runs on die
    floor(8 (k + 1/2) / K) (workgroup w = item // 4 runs on die w % 8), one
    of a row cut into fewer on a die of [floor(8k / K), ceil(8(k + 1) / K)),
    the pieces of one such span spread evenly over its dies; whole rows
    balance the dies' edges, and each die runs its items longest first."""
    c = synth.make_config("rmat_233k_115m", scale_down=64).csr
    kw = dict(segment_edges=S)
    plain, n_split, n_slot = fg.schedule_host(c.indptr, None, c.num_cols, 128, "plain", **kw)
    band, b_split, b_slot = fg.schedule_host(c.indptr, None, c.num_cols, 128, "gather",
                                             item_order=3, band_row_edges=-1, **kw)
    assert (n_split, n_slot) == (b_split, b_slot) and n_split > 0
    pad = band[:, 0] < 0
    assert np.all(band[pad, 1:] == [0, 0, -1])
    real = band[~pad]
    key = lambda a: a[np.lexsort((a[:, 3], a[:, 2], a[:, 1], a[:, 0]))]
    np.testing.assert_array_equal(key(real), key(plain))
    die = (np.nonzero(~pad)[0] // 4) % 8
    # slot ranges per split row: piece k of K
    slotted = real[:, 3] >= 0
    rows = real[slotted, 0]
    first = {}
    count = {}
    for r, sl in zip(rows, real[slotted, 3]):
        first[r] = min(first.get(r, sl), sl)
        count[r] = count.get(r, 0) + 1
    k = np.array([sl - first[r] for r, sl in zip(rows, real[slotted, 3])])
    K = np.array([count[r] for r in rows])
    banded = K >= 8
    np.testing.assert_array_equal(die[slotted][banded], ((16 * k + 8) // (2 * K))[banded])
    lo, hi = (8 * k) // K, -((-8 * (k + 1)) // K)
    d = die[slotted]
    assert np.all((d >= lo) & (d < hi))
    spans = set(zip(lo[~banded].tolist(), hi[~banded].tolist()))
    assert spans or S == 4096
    for a, b in spans:
        on = (lo == a) & (hi == b) & ~banded
        per = np.bincount(d[on] - a, minlength=b - a)
        assert per.max() - per.min() <= 1, (a, b, per)
    lens = real[:, 2] - real[:, 1]
    load = np.bincount(die, weights=lens, minlength=8)
    print("die loads", load)
    assert load.max() - load.min() <= max(lens.max(), 0.02 * load.sum())
    for x in range(8):
        assert np.all(np.diff(lens[die == x]) <= 0)


@pytest.mark.parametrize("T,cap", [(0, 0), (40, 0), (40, 5)])
def test_die_banded_cuts_mid_length_rows(T, cap):
    """item_order 3 cuts every row of more than band_row_edges edges (default
    256) into at least min(8, max_row_segments) even pieces, longer rows as
    before; with 8 pieces each goes to its own die.  The edge-softmax
    schedule is not affected."""
    c = synth.make_config("rmat_233k_115m", scale_down=64).csr
    S = 256
    kw = dict(segment_edges=S, max_row_segments=cap, band_row_edges=T)
    band, n_split, n_slot = fg.schedule_host(c.indptr, None, c.num_cols, 128, "gather",
                                             item_order=3, **kw)
    plain, *_ = fg.schedule_host(c.indptr, None, c.num_cols, 128, "plain", item_order=3, **kw)
    deg = np.diff(c.indptr)
    thr, cap_ = (T or 256), (cap or 128)
    base = np.minimum(np.maximum(-(-deg // S), 1), cap_)
    want = np.where(deg > thr, np.maximum(base, np.minimum(np.minimum(8, cap_), deg)), base)
    want[deg == 0] = 1
    pad = band[:, 0] < 0
    real = band[~pad]
    got = np.bincount(real[:, 0], minlength=len(deg))
    np.testing.assert_array_equal(got, want)
    assert np.sum(want[want > 1]) == n_slot and np.sum(want > 1) == n_split
    # pieces tile each row evenly: lengths differ by at most one
    order = np.lexsort((real[:, 1], real[:, 0]))
    r = real[order]
    lens = r[:, 2] - r[:, 1]
    for row in np.nonzero(want > 1)[0][:200]:
        L = lens[r[:, 0] == row]
        assert L.sum() == deg[row] and L.max() - L.min() <= 1
    # the plain schedule (same S here) keeps the length-only cut
    base[deg == 0] = 1
    np.testing.assert_array_equal(np.bincount(plain[plain[:, 0] >= 0, 0], minlength=len(deg)),
                                  base)
    # rows of exactly 8 pieces: one piece per die
    die = (np.nonzero(~pad)[0] // 4) % 8
    for row in np.nonzero(want == 8)[0][:200]:
        assert sorted(die[real[:, 0] == row].tolist()) == list(range(8))


def test_sddmm_schedule_on_spread_graphs():
    """With source slabs, a spread graph (no hot sources, no locality along
    row ids) and max_width >= 256, the plan's SDDMM schedule cuts every row
    where its sources change slab (slabs of at most ceil(num_cols / 16) ids),
    with no partial-result slots; otherwise it is the gather schedule."""
    rng = np.random.default_rng(5)
    n, m, d = 3000, 30000, 100
    dst = np.repeat(np.arange(n), d)
    src = rng.integers(0, m, size=n * d)
    c = synth.coo_to_csr(dst.astype(np.int64), src.astype(np.int64), n, m)
    kw = dict(source_slab_rows=4096)
    edge, e_split, e_slot = fg.schedule_host(c.indptr, c.indices, m, 256, "sddmm", **kw)
    gather, *_ = fg.schedule_host(c.indptr, c.indices, m, 256, "gather", **kw)
    assert e_split == 0 and e_slot == 0
    real = edge[edge[:, 0] >= 0]
    assert np.all(real[:, 3] == -1)
    cover = np.zeros(c.nnz, np.int32)
    for r, b, e, _ in real:
        assert c.indptr[r] <= b < e <= c.indptr[r + 1]
        cover[b:e] += 1
        s = c.indices[b:e]
        assert s.max() - s.min() < -(-m // 16)  # inside one slab
    assert np.all(cover == 1)
    pieces = np.bincount(real[:, 0], minlength=n)
    assert pieces.mean() > 8 and real.shape[0] > gather[gather[:, 0] >= 0].shape[0]
    # below 256 floats, or without slabs: the gather schedule serves the SDDMM
    for width, opts in ((128, kw), (256, {})):
        a, *_ = fg.schedule_host(c.indptr, c.indices, m, width, "sddmm", **opts)
        b, *_ = fg.schedule_host(c.indptr, c.indices, m, width, "gather", **opts)
        np.testing.assert_array_equal(a, b)
    # a power-law graph (hot sources) keeps the gather schedule too
    p = synth.make_config("rmat_233k_115m", scale_down=64).csr
    a, *_ = fg.schedule_host(p.indptr, p.indices, p.num_cols, 256, "sddmm", source_slab_rows=64)
    b, *_ = fg.schedule_host(p.indptr, p.indices, p.num_cols, 256, "gather", source_slab_rows=64)
    np.testing.assert_array_equal(a, b)
