"""Pins of the CPU oracle against things other than itself.

Each test ties one oracle function to a hand-worked example, a dense
brute-force definition (numpy / scipy / torch autograd in fp64), a closed form
or an invariant, so that a dropped term, a wrong sign or index, or a swapped
operand in the oracle fails at least one of them.  CPU only.
"""
import json
import os

import numpy as np
import pytest
import scipy.sparse as sp

import synth
from synth import CSR, coo_to_csr, csr_to_csc, csr_rows

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def O(oracle_lib):
    return oracle_lib


def _rand_graph(seed, n_rows=300, n_cols=None, e=3000, empty_frac=0.2):
    rng = np.random.default_rng(seed)
    n_cols = n_rows if n_cols is None else n_cols
    return synth.small_random_graph(rng, n_rows, n_cols, e, empty_frac)


def _dense_count(g: CSR) -> np.ndarray:
    a = np.zeros((g.num_rows, g.num_cols), np.float64)
    np.add.at(a, (csr_rows(g), g.indices), 1.0)
    return a


def _eids(g: CSR) -> np.ndarray:
    return np.arange(g.nnz, dtype=np.int64) if g.edge_ids is None else g.edge_ids.astype(np.int64)


# ---------------------------------------------------------------- golden


def _golden_graph():
    gd = json.load(open(os.path.join(GOLDEN, "hand_worked_4v.json")))
    c = gd["csr_rows_are_destinations"]
    g = CSR(4, 4, np.array(c["indptr"], np.int32), np.array(c["indices"], np.int32))
    # the CSR must be what the generation-order edge list sorts into
    e = np.array(gd["edges_src_to_dst_generation_order"])
    g2 = coo_to_csr(e[:, 1], e[:, 0], 4, 4)
    np.testing.assert_array_equal(g2.indptr, g.indptr)
    np.testing.assert_array_equal(g2.indices, g.indices)
    return gd, g


def test_golden_spmm(O):
    gd, g = _golden_graph()
    x = np.array(gd["x"], np.float32)
    w = np.array(gd["w"], np.float32)
    out = O.gspmm(g, x)
    np.testing.assert_array_equal(out, np.array(gd["copy_src_sum"]["value"], np.float32))
    out, arg = O.gspmm(g, x, red=O.RED_MAX)
    np.testing.assert_array_equal(out, np.array(gd["copy_src_max"]["value"], np.float32))
    np.testing.assert_array_equal(arg, np.array(gd["copy_src_max"]["arg"], np.int32))
    out = O.gspmm(g, x, msg=O.MSG_SRC_MUL_EDGE, edge_val=w)
    np.testing.assert_array_equal(out, np.array(gd["src_mul_edge_sum"]["value"], np.float32))
    out, arg = O.gspmm(g, x, msg=O.MSG_SRC_MUL_EDGE, red=O.RED_MAX, edge_val=w)
    np.testing.assert_array_equal(out, np.array(gd["src_mul_edge_max"]["value"], np.float32))
    np.testing.assert_array_equal(arg, np.array(gd["src_mul_edge_max"]["arg"], np.int32))


def test_golden_sddmm_softmax(O):
    gd, g = _golden_graph()
    x = np.array(gd["x"], np.float32)
    y = np.array(gd["y_dst"], np.float32)
    s = O.gsddmm(g, x, y)[:, 0]
    np.testing.assert_array_equal(s, np.array(gd["sddmm_dot_x_src_y_dst"]["value"], np.float32))
    ent = gd["edge_softmax_of_sddmm_leaky_0.2"]
    a = O.edge_softmax(g, s, leaky=True, slope=0.2)[:, 0]
    np.testing.assert_allclose(a, ent["value"], rtol=1e-6, atol=0)
    ent = gd["edge_softmax_of_sddmm_no_leaky"]
    a = O.edge_softmax(g, np.array(ent["scores_override"], np.float32), leaky=False)[:, 0]
    np.testing.assert_allclose(a, ent["value"], rtol=1e-6, atol=0)


# ---------------------------------------------------------------- gSpMM sum


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_spmm_sum_equals_dense_product(O, seed):
    g = _rand_graph(seed, n_rows=257, n_cols=190, e=4000)
    x = np.random.default_rng(100 + seed).standard_normal((g.num_cols, 19)).astype(np.float32)
    ref = _dense_count(g) @ x.astype(np.float64)
    out = O.gspmm(g, x)
    # one fp32 rounding of an fp64 sum: equal up to the last bit
    np.testing.assert_allclose(out, ref, rtol=2.5e-7, atol=1e-12)


@pytest.mark.parametrize("heads", [1, 4])
def test_spmm_weighted_sum_equals_scipy(O, heads):
    g = _rand_graph(7, n_rows=200, e=5000)
    rng = np.random.default_rng(8)
    dh = 6
    x = rng.standard_normal((g.num_cols, heads * dh)).astype(np.float32)
    w = rng.uniform(-2, 2, size=(g.nnz, heads)).astype(np.float32)
    out = O.gspmm(g, x, msg=O.MSG_SRC_MUL_EDGE, edge_val=w, heads=heads)
    for h in range(heads):
        # scipy may canonicalise (sum duplicates in) the arrays it is given: pass copies
        a = sp.csr_matrix((w[:, h].astype(np.float64), g.indices.copy(), g.indptr.copy()),
                          shape=(g.num_rows, g.num_cols))
        ref = a @ x[:, h * dh:(h + 1) * dh].astype(np.float64)
        absref = abs(a) @ np.abs(x[:, h * dh:(h + 1) * dh].astype(np.float64))
        # the oracle rounds each product to fp32 (<= 2^-24 relative per term)
        err = np.abs(out[:, h * dh:(h + 1) * dh] - ref)
        assert np.all(err <= 2.0 ** -23 * absref + 1e-30)


def test_spmm_integer_inputs_exact(O):
    g = _rand_graph(3, n_rows=500, e=20000, empty_frac=0.1)
    rng = np.random.default_rng(4)
    x = rng.integers(-8, 9, size=(g.num_cols, 5)).astype(np.float32)
    w = rng.integers(-3, 4, size=g.nnz).astype(np.float32)
    a = sp.csr_matrix((w.astype(np.int64), g.indices.copy(), g.indptr.copy()),
                      shape=(g.num_rows, g.num_cols))
    ref = a @ x.astype(np.int64)
    out = O.gspmm(g, x, msg=O.MSG_SRC_MUL_EDGE, edge_val=w)
    np.testing.assert_array_equal(out, ref.astype(np.float32))
    ref = _dense_count(g).astype(np.int64) @ x.astype(np.int64)
    np.testing.assert_array_equal(O.gspmm(g, x), ref.astype(np.float32))


def test_spmm_ones_give_degrees(O):
    g = _rand_graph(5, n_rows=400, e=6000, empty_frac=0.3)
    ones = np.ones((g.num_cols, 3), np.float32)
    out = O.gspmm(g, ones)
    np.testing.assert_array_equal(out[:, 0], g.degrees().astype(np.float32))
    # on the transposed graph the same features give out-degrees
    csc = csr_to_csc(g)
    out_t = O.gspmm(csc, np.ones((csc.num_cols, 2), np.float32))
    np.testing.assert_array_equal(out_t[:, 1],
                                  np.bincount(g.indices, minlength=g.num_cols).astype(np.float32))


# ---------------------------------------------------------------- gSpMM max / argmax


def _brute_max(g, x, w=None):
    F = x.shape[1]
    H = 1 if w is None else w.shape[1]
    dh = F // H
    eids = _eids(g)
    out = np.zeros((g.num_rows, F), np.float32)
    arg = np.full((g.num_rows, F), -1, np.int32)
    for v in range(g.num_rows):
        p = np.arange(g.indptr[v], g.indptr[v + 1])
        if p.size == 0:
            continue
        m = x[g.indices[p]].astype(np.float32)
        if w is not None:
            m = (np.repeat(w[eids[p]], dh, axis=1) * m).astype(np.float32)
        best = m.max(axis=0)
        for f in range(F):
            hit = eids[p][m[:, f] == best[f]]
            out[v, f] = best[f]
            arg[v, f] = hit.min()
    return out, arg


@pytest.mark.parametrize("transpose", [False, True])
def test_spmm_max_argmax_brute_force(O, transpose):
    g = _rand_graph(11, n_rows=120, e=2400, empty_frac=0.15)
    if transpose:
        g = csr_to_csc(g)  # edge ids are no longer positions
    rng = np.random.default_rng(12)
    x = rng.integers(-3, 4, size=(g.num_cols, 7)).astype(np.float32)  # many ties
    out, arg = O.gspmm(g, x, red=O.RED_MAX, nnz_total=g.nnz)
    bo, ba = _brute_max(g, x)
    np.testing.assert_array_equal(out, bo)
    np.testing.assert_array_equal(arg, ba)
    w = rng.integers(-2, 3, size=(g.nnz, 1)).astype(np.float32)
    out, arg = O.gspmm(g, x, msg=O.MSG_SRC_MUL_EDGE, red=O.RED_MAX, edge_val=w)
    bo, ba = _brute_max(g, x, w)
    np.testing.assert_array_equal(out, bo)
    np.testing.assert_array_equal(arg, ba)


def test_spmm_max_signed_zero_and_neg_inf(O):
    # row 0: -0.0 (e0) and +0.0 (e1) tie -> e0 wins and its bits are kept
    # row 1: +0.0 (e2) then -0.0 (e3) -> e2 wins, +0.0
    # row 2: all -inf -> value -inf, first edge id
    g = CSR(3, 4, np.array([0, 2, 4, 6], np.int32), np.array([0, 1, 1, 0, 2, 3], np.int32))
    x = np.array([[-0.0], [0.0], [-np.inf], [-np.inf]], np.float32)
    out, arg = O.gspmm(g, x, red=O.RED_MAX)
    assert np.signbit(out[0, 0]) and arg[0, 0] == 0
    assert not np.signbit(out[1, 0]) and arg[1, 0] == 2
    assert out[2, 0] == -np.inf and arg[2, 0] == 4


def test_spmm_max_all_equal_takes_first_edge(O):
    g = _rand_graph(13, n_rows=50, e=500, empty_frac=0.0)
    out, arg = O.gspmm(g, np.ones((g.num_cols, 2), np.float32), red=O.RED_MAX)
    deg = g.degrees()
    np.testing.assert_array_equal(arg[deg > 0, 0], g.indptr[:-1][deg > 0])
    np.testing.assert_array_equal(out[deg > 0], 1.0)
    np.testing.assert_array_equal(arg[deg == 0], -1)


# ---------------------------------------------------------------- gSDDMM


@pytest.mark.parametrize("heads,dh", [(1, 9), (3, 4)])
def test_sddmm_equals_masked_dense_product(O, heads, dh):
    g = _rand_graph(21, n_rows=150, n_cols=170, e=3000)
    rng = np.random.default_rng(22)
    xs = rng.standard_normal((g.num_cols, heads * dh)).astype(np.float32)
    xd = rng.standard_normal((g.num_rows, heads * dh)).astype(np.float32)
    out = O.gsddmm(g, xs, xd, heads=heads)
    dst, src = csr_rows(g), g.indices
    for h in range(heads):
        sl = slice(h * dh, (h + 1) * dh)
        dense = xd[:, sl].astype(np.float64) @ xs[:, sl].astype(np.float64).T  # [rows, cols]
        ref = dense[dst, src]
        np.testing.assert_allclose(out[:, h], ref, rtol=2.5e-7, atol=1e-12)


def test_sddmm_integer_exact_and_transpose_consistent(O):
    g = _rand_graph(23, n_rows=200, e=4000)
    rng = np.random.default_rng(24)
    x = rng.integers(-8, 9, size=(g.num_cols, 16)).astype(np.float32)
    y = rng.integers(-8, 9, size=(g.num_rows, 16)).astype(np.float32)
    out = O.gsddmm(g, x, y)[:, 0]
    ref = np.einsum("ek,ek->e", x[g.indices].astype(np.int64), y[csr_rows(g)].astype(np.int64))
    np.testing.assert_array_equal(out, ref.astype(np.float32))
    # same edge values through the transposed graph (rows = sources, by edge id)
    csc = csr_to_csc(g)
    out_t = O.gsddmm(csc, y, x, nnz_total=g.nnz)[:, 0]
    np.testing.assert_array_equal(out_t, out)


# ---------------------------------------------------------------- duality / adjoint


def test_adjoint_identity(O):
    """<dY, A X> = <A^T dY, X> = sum_e SDDMM(X, dY)[e] (Sec. II-A: the gradient of
    SpMM w.r.t. A is an SDDMM)."""
    rng = np.random.default_rng(31)
    g = synth.rmat_graph(np.random.SeedSequence(31), rng, 10, 1000, 20000)
    csc = csr_to_csc(g)
    x = rng.standard_normal((g.num_cols, 8)).astype(np.float32)
    dy = rng.standard_normal((g.num_rows, 8)).astype(np.float32)
    fwd = O.gspmm(g, x).astype(np.float64)
    bwd = O.gspmm(csc, dy).astype(np.float64)
    da = O.gsddmm(g, x, dy)[:, 0].astype(np.float64)
    a = np.sum(dy * fwd)
    b = np.sum(bwd * x)
    c = np.sum(da)
    scale = np.sum(np.abs(dy.astype(np.float64)) * (_dense_count(g) @ np.abs(x.astype(np.float64))))
    assert abs(a - b) <= 1e-6 * scale
    assert abs(a - c) <= 1e-6 * scale


def test_edge_weight_gradient_is_sddmm(O):
    """d<dY, A(w) X>/dw_e from torch autograd on a dense A(w) equals the SDDMM of
    X and dY at edge e."""
    torch = pytest.importorskip("torch")
    g = _rand_graph(41, n_rows=60, n_cols=70, e=700)
    rng = np.random.default_rng(42)
    x = rng.standard_normal((g.num_cols, 5)).astype(np.float32)
    dy = rng.standard_normal((g.num_rows, 5)).astype(np.float32)
    w = torch.ones(g.nnz, dtype=torch.float64, requires_grad=True)
    a = torch.zeros(g.num_rows, g.num_cols, dtype=torch.float64)
    idx = (torch.from_numpy(csr_rows(g).astype(np.int64)), torch.from_numpy(g.indices.astype(np.int64)))
    a = a.index_put(idx, w, accumulate=True)
    loss = (torch.from_numpy(dy).double() * (a @ torch.from_numpy(x).double())).sum()
    loss.backward()
    da = O.gsddmm(g, x, dy)[:, 0]
    np.testing.assert_allclose(da, w.grad.numpy(), rtol=2.5e-7, atol=1e-12)


def test_sddmm_gradient_is_spmm(O):
    """The gradient of an SDDMM is an SpMM (Sec. II-A): with scores
    s_e = Xs[src]·Xd[dst] and upstream gradient g_e,
    dL/dXs = SpMM over the transposed graph of Xd scaled by g (src_mul_edge, sum)."""
    torch = pytest.importorskip("torch")
    g = _rand_graph(43, n_rows=80, n_cols=90, e=900)
    csc = csr_to_csc(g)
    rng = np.random.default_rng(44)
    xs = rng.standard_normal((g.num_cols, 6)).astype(np.float32)
    xd = rng.standard_normal((g.num_rows, 6)).astype(np.float32)
    ge = rng.standard_normal(g.nnz).astype(np.float32)
    txs = torch.from_numpy(xs).double().requires_grad_(True)
    s = (txs[torch.from_numpy(g.indices.astype(np.int64))]
         * torch.from_numpy(xd).double()[torch.from_numpy(csr_rows(g).astype(np.int64))]).sum(1)
    (s * torch.from_numpy(ge).double()).sum().backward()
    dxs = O.gspmm(csc, xd, msg=O.MSG_SRC_MUL_EDGE, edge_val=ge.reshape(-1, 1))
    # the oracle rounds g_e * Xd to fp32 per term
    np.testing.assert_allclose(dxs, txs.grad.numpy(), rtol=1e-5, atol=1e-5)


# ---------------------------------------------------------------- edge softmax


@pytest.mark.parametrize("heads,leaky", [(1, True), (4, True), (2, False)])
def test_edge_softmax_matches_torch_softmax(O, heads, leaky):
    torch = pytest.importorskip("torch")
    g = _rand_graph(51, n_rows=100, e=2500, empty_frac=0.2)
    rng = np.random.default_rng(52)
    s = (3 * rng.standard_normal((g.nnz, heads))).astype(np.float32)
    out = O.edge_softmax(g, s, heads=heads, leaky=leaky, slope=0.2)
    ts = torch.from_numpy(s).double()
    if leaky:
        ts = torch.nn.functional.leaky_relu(ts, negative_slope=float(np.float32(0.2)))
    for v in range(g.num_rows):
        a, b = g.indptr[v], g.indptr[v + 1]
        if a == b:
            continue
        ref = torch.softmax(ts[a:b], dim=0).numpy()
        np.testing.assert_allclose(out[a:b], ref, rtol=1e-6, atol=1e-12)


def test_edge_softmax_invariants(O):
    g = _rand_graph(53, n_rows=300, e=5000, empty_frac=0.2)
    rng = np.random.default_rng(54)
    s = rng.standard_normal((g.nnz, 3)).astype(np.float32) * 10
    out = O.edge_softmax(g, s, heads=3)
    rs = np.add.reduceat(out.astype(np.float64), g.indptr[:-1][g.degrees() > 0], axis=0)
    np.testing.assert_allclose(rs, 1.0, rtol=0, atol=1e-6)
    # equal scores -> 1/deg; a single edge -> 1
    out = O.edge_softmax(g, np.full((g.nnz, 1), 0.7, np.float32))
    deg = np.repeat(g.degrees(), g.degrees())
    np.testing.assert_allclose(out[:, 0], 1.0 / deg, rtol=1e-7)
    # empty rows write nothing: untouched outputs stay NaN-filled
    assert not np.isnan(out).any()


def test_edge_softmax_through_edge_ids(O):
    """Softmax over the transposed graph normalises over out-edges, indexed by
    edge id; the result equals a softmax grouped by source vertex."""
    g = _rand_graph(55, n_rows=80, e=900, empty_frac=0.0)
    csc = csr_to_csc(g)
    s = np.random.default_rng(56).standard_normal((g.nnz, 1)).astype(np.float32)
    out = O.edge_softmax(csc, s, leaky=False, nnz_total=g.nnz)[:, 0]
    src = g.indices
    for u in np.unique(src)[:40]:
        m = src == u
        e = np.exp(s[m, 0].astype(np.float64) - s[m, 0].max())
        np.testing.assert_allclose(out[m], e / e.sum(), rtol=1e-6)


# ---------------------------------------------------------------- determinism / row selection


def test_thread_count_invariance_and_row_selection(O):
    g = _rand_graph(61, n_rows=700, e=30000, empty_frac=0.1)
    rng = np.random.default_rng(62)
    x = rng.standard_normal((g.num_cols, 12)).astype(np.float32)
    w = rng.random((g.nnz, 2)).astype(np.float32)
    for kw in (dict(), dict(msg=O.MSG_SRC_MUL_EDGE, edge_val=w, heads=2)):
        a1 = O.gspmm(g, x, threads=1, **kw)
        a8 = O.gspmm(g, x, threads=8, **kw)
        np.testing.assert_array_equal(a1, a8)
        rows = rng.choice(g.num_rows, 50, replace=False)
        np.testing.assert_array_equal(O.gspmm(g, x, rows=rows, **kw), a1[rows])
        m1, i1 = O.gspmm(g, x, red=O.RED_MAX, threads=1, **kw)
        m8, i8 = O.gspmm(g, x, red=O.RED_MAX, threads=8, **kw)
        np.testing.assert_array_equal(m1, m8)
        np.testing.assert_array_equal(i1, i8)
    s1 = O.gsddmm(g, x, x[: g.num_rows], threads=1)
    s8 = O.gsddmm(g, x, x[: g.num_rows], threads=8)
    np.testing.assert_array_equal(s1, s8)
    np.testing.assert_array_equal(O.edge_softmax(g, s1, threads=1), O.edge_softmax(g, s1, threads=8))


def test_invalid_arguments_rejected(O):
    g = _rand_graph(71, n_rows=10, e=30)
    x = np.ones((g.num_cols, 4), np.float32)
    with pytest.raises(ValueError):
        O.gspmm(g, x, msg=O.MSG_SRC_MUL_EDGE)  # missing edge values
    with pytest.raises(ValueError):
        O.gspmm(g, x, rows=[0, 10])  # row out of range
    bad = CSR(g.num_rows, g.num_cols, g.indptr, g.indices.copy())
    bad.indices[0] = g.num_cols  # source out of range
    with pytest.raises(ValueError):
        O.gspmm(bad, x)


# ---------------------------------------------------------------- backward of max and softmax


def test_golden_max_backward(O):
    gd, g = _golden_graph()
    x = np.array(gd["x"], np.float32)
    w = np.array(gd["w"], np.float32)
    c = gd["copy_src_max_backward"]
    go = np.array(c["grad_out"], np.float32)
    np.testing.assert_array_equal(O.gspmm_max_backward(g, x, go), np.array(c["grad_src"]))
    m = gd["src_mul_edge_max_backward"]
    dx, dw = O.gspmm_max_backward(g, x, go, msg=O.MSG_SRC_MUL_EDGE, edge_val=w.reshape(-1, 1),
                                  want_edge=True)
    np.testing.assert_array_equal(dx, np.array(m["grad_src"]))
    np.testing.assert_array_equal(dw[:, 0], np.array(m["grad_edge"]))


def test_golden_softmax_backward(O):
    gd, g = _golden_graph()
    b = gd["edge_softmax_backward"]
    s = np.array(b["scores"], np.float32).reshape(-1, 1)
    go = np.array(b["grad_out"], np.float32).reshape(-1, 1)
    ds = O.edge_softmax_backward(g, s, go, leaky=False)[:, 0]
    np.testing.assert_allclose(ds[:4], b["no_leaky_rows_0_1"]["value"], rtol=1e-6, atol=1e-12)
    ds = O.edge_softmax_backward(g, s, go, leaky=True, slope=0.2)[:, 0]
    np.testing.assert_allclose(ds[4:], b["leaky_0.2_row3"]["value"], rtol=1e-6, atol=1e-15)


def _max_autograd(torch, g, x, go, w=None, heads=1):
    """Reference gradient of sum(G * maxagg(messages)) by torch autograd (fp64):
    the messages of each row are laid out by increasing edge id in a padded
    [rows, slots, F] tensor, the kept edge is chosen by numpy's argmax on the
    fp32 messages (documented to return the first of equal maxima, i.e. the
    smallest edge id) and gathered, so autograd routes G to that edge."""
    eids = _eids(g)
    rows = csr_rows(g)
    deg = g.degrees()
    D = max(int(deg.max()), 1)
    F = x.shape[1]
    dh = F // heads
    order = np.lexsort((eids, rows))  # by row, then edge id
    slot = np.arange(g.nnz) - g.indptr[rows[order]]
    m32 = np.full((g.num_rows, D, F), -np.inf, np.float32)
    src = g.indices[order]
    e_sorted = eids[order]
    msg32 = x[src]
    if w is not None:
        msg32 = (np.repeat(w[e_sorted], dh, axis=1) * msg32).astype(np.float32)
    m32[rows[order], slot] = msg32
    pick = np.argmax(m32, axis=1)  # [rows, F]
    tx = torch.from_numpy(x).double().requires_grad_(True)
    tw = None if w is None else torch.from_numpy(w).double().requires_grad_(True)
    m = torch.zeros((g.num_rows, D, F), dtype=torch.float64)
    tmsg = tx[torch.from_numpy(src.astype(np.int64))]
    if tw is not None:
        tmsg = tw[torch.from_numpy(e_sorted.astype(np.int64))].repeat_interleave(dh, dim=1) * tmsg
    m = m.index_put((torch.from_numpy(rows[order].astype(np.int64)),
                     torch.from_numpy(slot.astype(np.int64))), tmsg)
    out = m.gather(1, torch.from_numpy(pick.astype(np.int64))[:, None, :])[:, 0, :]
    nonempty = torch.from_numpy((deg > 0).astype(np.float64))[:, None]
    (out * nonempty * torch.from_numpy(go).double()).sum().backward()
    return tx.grad.numpy(), (None if tw is None else tw.grad.numpy())


@pytest.mark.parametrize("weighted,heads,transpose,ties", [
    (False, 1, False, False), (False, 1, False, True), (True, 1, False, False),
    (True, 2, False, True), (False, 1, True, True), (True, 2, True, False)])
def test_max_backward_matches_torch_autograd(O, weighted, heads, transpose, ties):
    torch = pytest.importorskip("torch")
    g = _rand_graph(81, n_rows=120, n_cols=100, e=2400, empty_frac=0.2)
    nnz_total = g.nnz
    if transpose:
        g = csr_to_csc(g)
    rng = np.random.default_rng(82)
    F = 6
    if ties:  # small integers: many equal messages, the smallest edge id must win
        x = rng.integers(-2, 3, (g.num_cols, F)).astype(np.float32)
        w = rng.integers(1, 3, (nnz_total, heads)).astype(np.float32) if weighted else None
    else:
        x = rng.standard_normal((g.num_cols, F)).astype(np.float32)
        w = rng.random((nnz_total, heads)).astype(np.float32) + 0.5 if weighted else None
    go = rng.standard_normal((g.num_rows, F)).astype(np.float32)
    ref_x, ref_w = _max_autograd(torch, g, x, go, w, heads)
    if weighted:
        dx, dw = O.gspmm_max_backward(g, x, go, msg=O.MSG_SRC_MUL_EDGE, edge_val=w, heads=heads,
                                      nnz_total=nnz_total, want_edge=True)
        np.testing.assert_allclose(dw, ref_w, rtol=1e-6, atol=1e-12)
    else:
        dx = O.gspmm_max_backward(g, x, go, nnz_total=nnz_total)
    np.testing.assert_allclose(dx, ref_x, rtol=1e-6, atol=1e-12)


def test_max_backward_conserves_gradient_and_threads(O):
    """copy_src: every non-empty row sends each G[v, k] to exactly one source,
    so column sums of dX equal those of G over non-empty rows; row selection
    keeps only the selected rows' contributions; threads do not matter."""
    g = _rand_graph(83, n_rows=400, e=9000, empty_frac=0.15)
    rng = np.random.default_rng(84)
    x = rng.standard_normal((g.num_cols, 5)).astype(np.float32)
    go = rng.integers(-8, 9, (g.num_rows, 5)).astype(np.float32)
    dx = O.gspmm_max_backward(g, x, go, threads=1)
    np.testing.assert_array_equal(dx.sum(0), go[g.degrees() > 0].sum(0))
    np.testing.assert_array_equal(dx, O.gspmm_max_backward(g, x, go, threads=8))
    rows = np.flatnonzero(np.arange(g.num_rows) % 3 == 0)
    go_sel = np.zeros_like(go)
    go_sel[rows] = go[rows]
    np.testing.assert_array_equal(O.gspmm_max_backward(g, x, go, rows=rows),
                                  O.gspmm_max_backward(g, x, go_sel))


@pytest.mark.parametrize("heads,leaky,transpose", [(1, True, False), (3, True, False),
                                                   (2, False, False), (1, True, True)])
def test_softmax_backward_matches_torch_autograd(O, heads, leaky, transpose):
    torch = pytest.importorskip("torch")
    g = _rand_graph(85, n_rows=150, e=3000, empty_frac=0.2)
    nnz_total = g.nnz
    if transpose:
        g = csr_to_csc(g)
    rng = np.random.default_rng(86)
    s = (2 * rng.standard_normal((nnz_total, heads))).astype(np.float32)
    s[rng.random((nnz_total, heads)) < 0.05] = 0.0  # the leaky kink: slope at exactly 0
    go = rng.standard_normal((nnz_total, heads)).astype(np.float32)
    ds = O.edge_softmax_backward(g, s, go, heads=heads, leaky=leaky, slope=0.2,
                                 nnz_total=nnz_total)
    ts = torch.from_numpy(s).double().requires_grad_(True)
    t = torch.nn.functional.leaky_relu(ts, negative_slope=float(np.float32(0.2))) if leaky else ts
    eids = _eids(g)
    loss = 0
    for v in range(g.num_rows):
        a, b = g.indptr[v], g.indptr[v + 1]
        if a == b:
            continue
        idx = torch.from_numpy(eids[a:b])
        loss = loss + (torch.softmax(t[idx], dim=0) * torch.from_numpy(go).double()[idx]).sum()
    loss.backward()
    np.testing.assert_allclose(ds, ts.grad.numpy(), rtol=1e-5, atol=1e-9)


def test_softmax_backward_invariants(O):
    g = _rand_graph(87, n_rows=300, e=6000, empty_frac=0.2)
    rng = np.random.default_rng(88)
    s = (3 * rng.standard_normal((g.nnz, 2))).astype(np.float32)
    go = rng.standard_normal((g.nnz, 2)).astype(np.float32)
    ds = O.edge_softmax_backward(g, s, go, heads=2, leaky=False, threads=1)
    nz = g.degrees() > 0
    rs = np.add.reduceat(ds.astype(np.float64), g.indptr[:-1][nz], axis=0)
    np.testing.assert_allclose(rs, 0.0, atol=1e-6)  # softmax outputs sum to one
    # a gradient constant over each row changes nothing
    const = np.repeat(rng.standard_normal(g.num_rows).astype(np.float32), g.degrees())
    ds0 = O.edge_softmax_backward(g, s, np.stack([const, const], 1), heads=2, leaky=False)
    np.testing.assert_allclose(ds0, 0.0, atol=1e-6)
    np.testing.assert_array_equal(ds, O.edge_softmax_backward(g, s, go, heads=2, leaky=False,
                                                              threads=8))
    rows = rng.choice(g.num_rows, 40, replace=False)
    part = O.edge_softmax_backward(g, s, go, heads=2, leaky=False, rows=rows)
    sel = np.concatenate([np.arange(g.indptr[r], g.indptr[r + 1]) for r in rows])
    np.testing.assert_array_equal(part[sel], ds[sel])


def test_backward_invalid_arguments_rejected(O):
    g = _rand_graph(89, n_rows=10, e=30)
    x = np.ones((g.num_cols, 4), np.float32)
    go = np.ones((g.num_rows, 4), np.float32)
    with pytest.raises(ValueError):
        O.gspmm_max_backward(g, x, go, want_edge=True)  # copy_src has no edge values
    with pytest.raises(ValueError):
        O.gspmm_max_backward(g, x, go, msg=O.MSG_SRC_MUL_EDGE)  # missing edge values
    dup = CSR(g.num_rows, g.num_cols, g.indptr, g.indices, np.zeros(g.nnz, np.int32))
    with pytest.raises(ValueError):
        O.gspmm_max_backward(dup, x, go, nnz_total=g.nnz)  # edge ids not distinct


# ---------------------------------------------------------------- MLP aggregation


def test_golden_mlp_aggregate(O):
    gd, g = _golden_graph()
    x = np.array(gd["x"], np.float32)
    m = gd["mlp_aggregate"]
    out, arg = O.mlp_aggregate(g, x, x, np.array(m["w"], np.float32))
    np.testing.assert_array_equal(out, np.array(m["value"]))
    np.testing.assert_array_equal(arg, np.array(m["arg"]))


def _mlp_brute(g, xs, xd, w):
    """Every message materialised with numpy (fp64 matmul), laid out per row by
    increasing edge id, max by numpy's argmax (first of equal maxima)."""
    eids = _eids(g)
    rows = csr_rows(g)
    msg = np.maximum((xs[g.indices].astype(np.float64) + xd[rows].astype(np.float64))
                     @ w.astype(np.float64), 0.0)
    D = max(int(g.degrees().max()), 1)
    order = np.lexsort((eids, rows))
    slot = np.arange(g.nnz) - g.indptr[rows[order]]
    pad = np.full((g.num_rows, D, w.shape[1]), -np.inf)
    ide = np.full((g.num_rows, D), -1, np.int64)
    pad[rows[order], slot] = msg[order]
    ide[rows[order], slot] = eids[order]
    k = np.argmax(pad, axis=1)
    out = np.take_along_axis(pad, k[:, None, :], 1)[:, 0, :]
    arg = np.take_along_axis(ide, k, 1)
    empty = g.degrees() == 0
    out[empty] = 0.0
    arg[empty] = -1
    return out, arg


@pytest.mark.parametrize("d_in,d_out,transpose", [(8, 16, False), (3, 5, False), (8, 7, True)])
def test_mlp_aggregate_brute_force(O, d_in, d_out, transpose):
    g = _rand_graph(91, n_rows=150, n_cols=130, e=2500, empty_frac=0.15)
    nnz_total = g.nnz
    if transpose:
        g = csr_to_csc(g)
    rng = np.random.default_rng(92)
    xs = rng.standard_normal((g.num_cols, d_in)).astype(np.float32)
    xd = rng.standard_normal((g.num_rows, d_in)).astype(np.float32)
    w = rng.standard_normal((d_in, d_out)).astype(np.float32)
    out, arg = O.mlp_aggregate(g, xs, xd, w, nnz_total=nnz_total)
    ref, rarg = _mlp_brute(g, xs, xd, w)
    np.testing.assert_allclose(out, ref, rtol=1e-6, atol=0)
    np.testing.assert_array_equal(arg, rarg)  # ties only at exact zeros (ReLU)
    assert (out == 0).any() and (arg[g.degrees() > 0] >= 0).all()


def test_mlp_aggregate_identity_weight_is_shifted_max(O):
    """W = I: m_e = relu(x_u + x_v), so out[v] = relu(max_u x_u + x_v) with the
    gSpMM-max edge where that is positive."""
    g = _rand_graph(93, n_rows=200, e=3000, empty_frac=0.1)
    rng = np.random.default_rng(94)
    x = rng.standard_normal((g.num_cols, 6)).astype(np.float32)
    out, arg = O.mlp_aggregate(g, x, x[: g.num_rows], np.eye(6, dtype=np.float32))
    mx, marg = O.gspmm(g, x, red=O.RED_MAX)
    shifted = mx.astype(np.float64) + x[: g.num_rows].astype(np.float64)
    ne = (g.degrees() > 0)[:, None]
    np.testing.assert_array_equal(out, np.where(ne, np.maximum(shifted, 0), 0).astype(np.float32))
    pos = ne & (shifted > 0)
    np.testing.assert_array_equal(arg[pos], marg[pos])


def test_mlp_aggregate_homogeneous_and_threads(O):
    g = _rand_graph(95, n_rows=120, e=2000)
    rng = np.random.default_rng(96)
    x = rng.standard_normal((g.num_cols, 8)).astype(np.float32)
    w = rng.standard_normal((8, 12)).astype(np.float32)
    o1, a1 = O.mlp_aggregate(g, x, x[: g.num_rows], w, threads=1)
    o2, a2 = O.mlp_aggregate(g, x, x[: g.num_rows], 2 * w, threads=8)
    np.testing.assert_array_equal(o2, 2 * o1)  # relu is positively homogeneous
    np.testing.assert_array_equal(a2, a1)
    rows = np.array([0, 5, 17, 119])
    o3, a3 = O.mlp_aggregate(g, x, x[: g.num_rows], w, rows=rows)
    np.testing.assert_array_equal(o3, o1[rows])
    np.testing.assert_array_equal(a3, a1[rows])


# ---------------------------------------------------------------- dense transform


def test_golden_dense_matmul(O):
    """Hand-worked product with a square, non-symmetric W (a transposed W is
    a different, also hand-worked, result)."""
    gd = json.load(open(os.path.join(GOLDEN, "dense_matmul_2x3x3.json")))
    x, w = np.array(gd["x"], np.float32), np.array(gd["w"], np.float32)
    y = O.dense_matmul(x, w)
    assert y.dtype == np.float64 and y.shape == (2, 3)
    np.testing.assert_array_equal(y, np.array(gd["y"]))
    assert not np.array_equal(y, np.array(gd["y_with_w_transposed"]))


def test_dense_matmul_against_library_and_special_cases(O):
    rng = np.random.default_rng(97)
    x = rng.standard_normal((37, 8)).astype(np.float32)
    w = rng.standard_normal((8, 13)).astype(np.float32)
    y = O.dense_matmul(x, w, threads=3)
    # a library product of the same fp32 inputs in fp64 (fp32 x fp32 products
    # are exact in fp64, so only the order of 8 additions may differ)
    np.testing.assert_allclose(y, x.astype(np.float64) @ w.astype(np.float64), rtol=1e-14,
                               atol=1e-14)
    np.testing.assert_array_equal(O.dense_matmul(x, np.eye(8, dtype=np.float32)), x)
    # a one-hot weight column picks one input column
    e3 = np.zeros((8, 1), np.float32)
    e3[3, 0] = 1.0
    np.testing.assert_array_equal(O.dense_matmul(x, e3)[:, 0], x[:, 3])
    # linearity in x: rows are independent
    np.testing.assert_array_equal(O.dense_matmul(x[5:9], w), y[5:9])
    assert O.dense_matmul(np.zeros((0, 8), np.float32), w).shape == (0, 13)


# ---------------------------------------------------------------- NaN in max


def test_max_nan_message_counts_as_minus_inf(O):
    """The library's reading for NaN messages (the paper defines none): a NaN
    competes as -inf, so it never beats a number, and a row of NaN / -inf
    messages reports -inf with its smallest edge id.  Worked by hand."""
    nan, inf = np.float32(np.nan), np.float32(np.inf)
    x = np.array([[nan], [5.0], [-inf]], np.float32)
    # row 0: NaN, 5 | row 1: NaN, NaN | row 2: NaN, -inf | row 3: -inf, NaN
    g = CSR(4, 3, np.array([0, 2, 4, 6, 8], np.int32),
            np.array([0, 1, 0, 0, 0, 2, 2, 0], np.int32))
    out, arg = O.gspmm(g, x, red=O.RED_MAX)
    np.testing.assert_array_equal(out[:, 0], [5.0, -inf, -inf, -inf])
    np.testing.assert_array_equal(arg[:, 0], [1, 2, 4, 6])
    # a weighted message 0 * inf is NaN as well
    xw = np.array([[inf], [1.0], [-2.0]], np.float32)
    w = np.array([0.0, 1.0, 0.0, 3.0, 1.0, 1.0, 1.0, 1.0], np.float32)
    out, arg = O.gspmm(g, xw, msg=O.MSG_SRC_MUL_EDGE, edge_val=w, red=O.RED_MAX)
    # row 0: NaN, 1 -> 1 (e1) | row 1: NaN, 3*inf -> inf (e3) | row 2: inf, -2 -> inf (e4)
    # row 3: -2, inf -> inf (e7)
    np.testing.assert_array_equal(out[:, 0], [1.0, inf, inf, inf])
    np.testing.assert_array_equal(arg[:, 0], [1, 3, 4, 7])
