"""Input generators: structure, exact sizes, determinism (CPU only)."""
import numpy as np
import pytest

import synth
from synth import check_csr, csr_rows, csr_to_csc, make_config, sha256


def test_tiny_uniform_shape_and_determinism():
    a = make_config("tiny_uniform_1k")
    b = make_config("tiny_uniform_1k")
    check_csr(a.csr)
    assert a.csr.num_rows == 1024 and a.csr.nnz == 16384
    assert a.arrays["x"].shape == (1024, 32) and a.arrays["x"].dtype == np.float32
    assert np.all(a.arrays["x"] >= -1) and np.all(a.arrays["x"] < 1)
    for k in ("x",):
        assert sha256(a.arrays[k]) == sha256(b.arrays[k])
    assert sha256(a.csr.indices) == sha256(b.csr.indices)
    # rows sorted by source inside each row
    d = np.diff(a.csr.indices.astype(np.int64))
    starts = a.csr.indptr[1:-1]
    d[starts[starts < d.size + 1] - 1] = 0
    assert np.all(d >= 0)


def test_fixed_indegree_rows():
    w = make_config("uniform_deg100_100k", d=32, scale_down=20)
    check_csr(w.csr)
    assert np.all(w.csr.degrees() == 100)
    assert w.arrays["x"].shape == (5000, 32)
    # a different width draws from its own stream
    w2 = make_config("uniform_deg100_100k", d=64, scale_down=20)
    assert sha256(w.csr.indices) == sha256(w2.csr.indices)


def test_clustered_degree_and_locality():
    w = make_config("clustered_133k_deg300", scale_down=50)
    check_csr(w.csr)
    n = w.csr.num_rows
    assert np.all(w.csr.degrees() == 300)
    dst = csr_rows(w.csr).astype(np.int64)
    src = w.csr.indices.astype(np.int64)
    same = (100 * dst) // n == (100 * src) // n
    # 270 of 300 in-community, plus the uniform ones that happen to land inside
    frac = same.mean()
    assert 0.9 <= frac <= 0.9 + 0.1 * 0.05
    assert w.arrays["x"].shape == (n, 8, 16)


def test_rmat_exact_edges_no_self_loops_and_skew():
    w = make_config("rmat_233k_115m", scale_down=64)
    check_csr(w.csr)
    assert w.csr.nnz == 114_600_000 // 64
    assert not np.any(csr_rows(w.csr) == w.csr.indices)
    deg = w.csr.degrees()
    assert deg.max() > 50 * deg.mean()  # power-law hub
    assert w.arrays["w"].min() > 0 and w.arrays["w"].max() <= 1
    w2 = make_config("rmat_233k_115m", scale_down=64)
    assert sha256(w.csr.indices) == sha256(w2.csr.indices)


def test_training_workload_csc_is_transpose():
    w = make_config("rmat_1m_33m_train", d=8, scale_down=256)
    csr, csc = w.csr, w.csc
    check_csr(csr)
    check_csr(csc, nnz_total=csr.nnz)
    assert csr.nnz == (1 << 25) // 256
    e = csc.edge_ids.astype(np.int64)
    assert np.array_equal(np.sort(e), np.arange(csr.nnz))
    # CSC row u, entry p  <->  CSR edge e = edge_ids[p] with src u and dst indices[p]
    np.testing.assert_array_equal(csr.indices[e], csr_rows(csc))
    np.testing.assert_array_equal(csr_rows(csr)[e], csc.indices)


def test_check_csr_rejects_bad_graphs():
    g = synth.small_random_graph(np.random.default_rng(0), 10, 10, 50)
    check_csr(g)
    bad = synth.CSR(g.num_rows, g.num_cols, g.indptr.copy(), g.indices.copy())
    bad.indices[3] = 10
    with pytest.raises(ValueError):
        check_csr(bad)
    bad = synth.CSR(g.num_rows, g.num_cols, g.indptr.copy(), g.indices.copy())
    bad.indptr[2], bad.indptr[3] = bad.indptr[3] + 1, bad.indptr[2]
    with pytest.raises(ValueError):
        check_csr(bad)
    t = csr_to_csc(g)
    bad = synth.CSR(t.num_rows, t.num_cols, t.indptr, t.indices, t.edge_ids.copy())
    bad.edge_ids[0] = g.nnz
    with pytest.raises(ValueError):
        check_csr(bad, nnz_total=g.nnz)


def test_two_class_degrees():
    """rand-100K shape: a fifth of the vertices hot with ~20x the degree of the
    rest, both in and out; exact edge count; deterministic."""
    w = synth.make_config("rand_100k_48m", d=16, scale_down=20)
    g = w.csr
    assert g.num_rows == 5000 and g.nnz == 2_400_000
    indeg = g.degrees()
    outdeg = np.bincount(g.indices, minlength=g.num_cols)
    for deg in (indeg, outdeg):
        top = np.sort(deg)[::-1]
        assert abs(top[:1000].mean() - 2000) < 60 and abs(top[1000:].mean() - 100) < 5
    w2 = synth.make_config("rand_100k_48m", d=16, scale_down=20)
    np.testing.assert_array_equal(w2.csr.indices, g.indices)
    np.testing.assert_array_equal(w2.arrays["x"], w.arrays["x"])
