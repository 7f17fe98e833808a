"""fg_gspmm_noalloc (the allocation-free gSpMM) against fg_gspmm, through the
C ABI.  With the same plan both run the same kernels in the same order, so
their results must agree bitwise; the first call of each case is also checked
against the oracle.  The fixed scratch keeps the previous call's contents, so
every case runs two calls in a row, the second on a smaller input."""
import numpy as np
import pytest
import torch

import oracle as O
import synth

pytestmark = pytest.mark.gpu

fg = None


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


def _both(G, x, plan, reduce, edge=None, heads=1):
    """One call of each entry point; returns (noalloc result, gspmm result)
    as host arrays (max: values as uint32 bits and edge ids)."""
    msg = "copy_src" if edge is None else "src_mul_edge"
    F = int(np.prod(x.shape[1:]))
    tx = dev(x)
    te = None if edge is None else dev(edge)
    out = torch.full((G.num_rows, F), float("nan"), device="cuda")
    arg = torch.full((G.num_rows, F), -7, dtype=torch.int32, device="cuda") \
        if reduce == "max" else None
    r_na = fg.gspmm_noalloc(G, tx.reshape(G.num_cols, F), out, arg, edge=te, msg=msg,
                            reduce=reduce, heads=heads, plan=plan)
    r_ref = fg.gspmm(G, tx.reshape(G.num_cols, F), te, msg=msg, reduce=reduce, heads=heads,
                     plan=plan)
    if reduce == "max":
        return (host(r_na[0]).view(np.uint32), host(r_na[1])), \
               (host(r_ref[0]).view(np.uint32), host(r_ref[1]))
    return (host(r_na).view(np.uint32),), (host(r_ref).view(np.uint32),)


def _against_oracle(csr, x, got, reduce, edge=None, heads=1):
    F = int(np.prod(x.shape[1:]))
    x2 = x.reshape(csr.num_cols, F)
    kw = dict(msg=O.MSG_COPY_SRC if edge is None else O.MSG_SRC_MUL_EDGE, heads=heads,
              edge_val=None if edge is None else edge.reshape(-1, heads))
    if reduce == "max":
        ro, ra = O.gspmm(csr, x2, red=O.RED_MAX, **kw)
        np.testing.assert_array_equal(got[0], ro.view(np.uint32))
        np.testing.assert_array_equal(got[1], ra)
        return
    ro, norm = O.gspmm(csr, x2, red=O.RED_SUM, with_norm=True, **kw)
    y = got[0].view(np.float32).astype(np.float64)
    n = np.maximum(csr.degrees(), 1)[:, None].astype(np.float64)
    bound = 1e-5 * np.sqrt(n) * np.maximum(np.abs(ro), norm)
    assert (np.abs(y - ro) <= bound).all()


def _case(csr, F, seg, reduce, weighted, heads, seed, check_oracle):
    rng = np.random.default_rng(seed)
    G = fg.Graph.from_csr(csr)
    plan = fg.Plan(G, max_width=F, segment_edges=seg)
    info = plan.info()
    say("noalloc rows=%d nnz=%d F=%d H=%d seg=%d reduce=%s weighted=%s slots=%d split=%d" % (
        csr.num_rows, csr.nnz, F, heads, seg, reduce, weighted, info["num_slots"],
        info["num_split_rows"]))
    assert info["num_split_rows"] > 0, "the case must exercise the scratch"
    x = rng.standard_normal((csr.num_cols, F)).astype(np.float32)
    edge = rng.random(csr.nnz * heads, dtype=np.float32).reshape(csr.nnz, heads) \
        if weighted else None
    if heads == 1 and edge is not None:
        edge = edge[:, 0].copy()
    got, ref = _both(G, x, plan, reduce, edge, heads)
    for a, b in zip(got, ref):
        np.testing.assert_array_equal(a, b)
    if check_oracle:
        _against_oracle(csr, x, got, reduce, edge, heads)
    plan.close()


@pytest.mark.parametrize("reduce,weighted,heads", [
    ("sum", False, 1), ("sum", True, 1), ("max", False, 1), ("max", True, 1), ("sum", True, 4)])
def test_noalloc_matches_gspmm_two_calls(reduce, weighted, heads):
    # first call: a power-law graph with a 500+ edge hub, float4 rows of 64,
    # 16-edge pieces (many slots)
    big = synth.rmat_graph(np.random.SeedSequence(77), np.random.default_rng(77), 11, 2000, 40000)
    _case(big, 64, 16, reduce, weighted, heads, seed=1, check_oracle=True)
    # second call, smaller: the tiny uniform graph, odd width (scalar lanes)
    small = synth.make_config("tiny_uniform_1k").csr
    _case(small, 8 * heads if heads > 1 else 7, 5, reduce, weighted, heads, seed=2,
          check_oracle=True)


def test_noalloc_without_splits_and_without_plan():
    csr = synth.make_config("tiny_uniform_1k").csr
    G = fg.Graph.from_csr(csr)
    x = np.random.default_rng(3).standard_normal((csr.num_cols, 32)).astype(np.float32)
    for plan in (None, fg.Plan(G, max_width=32)):  # default plan: rows of 16 edges stay whole
        if plan is not None:
            assert plan.info()["num_split_rows"] == 0
        for reduce in ("sum", "max"):
            say("noalloc no-split plan=%s reduce=%s" % (plan is not None, reduce))
            got, ref = _both(G, x, plan, reduce)
            for a, b in zip(got, ref):
                np.testing.assert_array_equal(a, b)


def test_noalloc_rejects_beyond_scratch():
    # one row of 9,000 edges cut into single-edge pieces: 9,000 slots; at
    # F = 1,024 the sum partials need 36.9 MB > 32 MiB
    n = 9000
    csr = synth.coo_to_csr(np.zeros(n, np.int64), np.arange(n) % 64, 1, 64)
    G = fg.Graph.from_csr(csr)
    plan = fg.Plan(G, max_width=1024, segment_edges=1, max_row_segments=n)
    assert plan.info()["num_slots"] == n
    x = torch.zeros((64, 1024), device="cuda")
    out = torch.full((1, 1024), 3.0, device="cuda")
    say("noalloc rejects %d slots x 1024" % n)
    with pytest.raises(fg.FgError) as e:
        fg.gspmm_noalloc(G, x, out, plan=plan)
    assert e.value.status == fg.FG_ERR_SCRATCH_LIMIT
    assert (host(out) == 3.0).all(), "a rejected call must write nothing"
    # half the width fits (9,000 x 512 x 4 bytes = 18.4 MB) and runs
    x2 = torch.ones((64, 512), device="cuda")
    out2 = torch.empty((1, 512), device="cuda")
    fg.gspmm_noalloc(G, x2, out2, plan=plan)
    assert (host(out2) == float(n)).all()
    plan.close()
