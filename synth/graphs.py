"""Seeded graph and feature generators (input generation only).

Conventions shared by every consumer:

* A graph is stored as CSR whose rows are DESTINATION vertices; ``indices``
  holds the source vertex of each stored edge.  Row ``v`` therefore lists the
  in-neighbours of ``v``, the set N(v) that the vertex-wise message-passing
  update (Sec. II-A, Eq. 1) reduces over.
* Within a row, edges are sorted by source id; the edge id of an edge is its
  position in this CSR (sort on (dst, src) of the generation order, stable).
* The transposed graph (CSC of the same adjacency, rows = source vertices)
  carries ``edge_ids`` = the CSR position of every edge, so edge data stays
  indexed by the one edge id.
* Everything is drawn from ``numpy.random.default_rng`` children of one
  ``SeedSequence``; separate children are used for structure, features,
  edge weights and output gradients so that one array can change without
  moving the others.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import Dict, Optional, Sequence

import numpy as np

# --------------------------------------------------------------------------
# containers
# --------------------------------------------------------------------------


@dataclasses.dataclass
class CSR:
    num_rows: int
    num_cols: int
    indptr: np.ndarray  # int32 [num_rows + 1]
    indices: np.ndarray  # int32 [nnz]
    edge_ids: Optional[np.ndarray] = None  # int32 [nnz] or None (= position)

    @property
    def nnz(self) -> int:
        return int(self.indptr[-1]) if self.indptr.size else 0

    def degrees(self) -> np.ndarray:
        return np.diff(self.indptr.astype(np.int64))


@dataclasses.dataclass
class Workload:
    name: str
    csr: CSR
    csc: Optional[CSR]
    arrays: Dict[str, np.ndarray]
    meta: Dict[str, object]


def sha256(a: np.ndarray) -> str:
    a = np.ascontiguousarray(a)
    h = hashlib.sha256()
    h.update(str(a.dtype).encode())
    h.update(str(a.shape).encode())
    h.update(a.view(np.uint8).reshape(-1).data)
    return h.hexdigest()


# --------------------------------------------------------------------------
# layout helpers (structure only)
# --------------------------------------------------------------------------


def _indptr_from_sorted_rows(rows_sorted: np.ndarray, num_rows: int) -> np.ndarray:
    counts = np.bincount(rows_sorted, minlength=num_rows).astype(np.int64)
    indptr = np.zeros(num_rows + 1, dtype=np.int64)
    np.cumsum(counts, out=indptr[1:])
    if indptr[-1] > np.iinfo(np.int32).max:
        raise ValueError("nnz exceeds int32")
    return indptr.astype(np.int32)


def coo_to_csr(dst: np.ndarray, src: np.ndarray, num_rows: int, num_cols: int) -> CSR:
    """Sort edges by (dst, src); the resulting position is the edge id."""
    dst = np.asarray(dst, dtype=np.int64)
    src = np.asarray(src, dtype=np.int64)
    key = dst * np.int64(num_cols) + src
    # equal keys are the same (dst, src) pair, so any sort yields the same CSR
    key.sort()
    rows = (key // num_cols).astype(np.int64)
    cols = (key % num_cols).astype(np.int32)
    indptr = _indptr_from_sorted_rows(rows, num_rows)
    return CSR(num_rows, num_cols, indptr, cols, None)


def csr_rows(csr: CSR) -> np.ndarray:
    """Destination (row) of every stored edge, in CSR order."""
    return np.repeat(np.arange(csr.num_rows, dtype=np.int32), csr.degrees())


def csr_to_csc(csr: CSR) -> CSR:
    """Transpose: rows become source vertices, ``edge_ids`` keep CSR positions.

    Within each CSC row the edges appear in increasing CSR position (a stable
    sort on the source id), so their edge ids are increasing too.
    """
    if csr.edge_ids is not None:
        raise ValueError("csr_to_csc expects a CSR whose edge ids are positions")
    order = np.argsort(csr.indices, kind="stable").astype(np.int32)
    src_sorted = csr.indices[order]
    indptr = _indptr_from_sorted_rows(src_sorted.astype(np.int64), csr.num_cols)
    dst_of_edge = csr_rows(csr)
    return CSR(csr.num_cols, csr.num_rows, indptr, dst_of_edge[order], order)


def check_csr(csr: CSR, nnz_total: Optional[int] = None) -> None:
    """Raise ValueError unless ``csr`` is a structurally valid graph."""
    ip = csr.indptr
    if ip.dtype != np.int32 or csr.indices.dtype != np.int32:
        raise ValueError("indptr and indices must be int32")
    if ip.shape != (csr.num_rows + 1,):
        raise ValueError("indptr has the wrong length")
    if ip[0] != 0:
        raise ValueError("indptr[0] must be 0")
    if csr.num_rows and np.any(np.diff(ip.astype(np.int64)) < 0):
        raise ValueError("indptr must be nondecreasing")
    nnz = int(ip[-1])
    if csr.indices.shape != (nnz,):
        raise ValueError("indices must have indptr[-1] entries")
    if nnz and (csr.indices.min() < 0 or csr.indices.max() >= csr.num_cols):
        raise ValueError("indices out of range")
    if csr.edge_ids is not None:
        if csr.edge_ids.dtype != np.int32 or csr.edge_ids.shape != (nnz,):
            raise ValueError("edge_ids must be int32 [nnz]")
        hi = nnz if nnz_total is None else nnz_total
        if nnz and (csr.edge_ids.min() < 0 or csr.edge_ids.max() >= hi):
            raise ValueError("edge_ids out of range")


# --------------------------------------------------------------------------
# structure generators
# --------------------------------------------------------------------------


def uniform_graph(rng: np.random.Generator, n: int, e: int) -> CSR:
    """src, dst i.i.d. uniform on [0, n); duplicates and self-loops kept."""
    dst = rng.integers(0, n, size=e, dtype=np.int64)
    src = rng.integers(0, n, size=e, dtype=np.int64)
    return coo_to_csr(dst, src, n, n)


def fixed_indegree_graph(rng: np.random.Generator, n: int, deg: int) -> CSR:
    """Every vertex gets exactly ``deg`` sources uniform on [0, n), with
    replacement (Table V's uniform-graph family at fixed density)."""
    src = rng.integers(0, n, size=(n, deg), dtype=np.int32)
    src.sort(axis=1)
    indptr = (np.arange(n + 1, dtype=np.int64) * deg).astype(np.int32)
    return CSR(n, n, indptr, src.reshape(-1), None)


def clustered_graph(rng: np.random.Generator, n: int, communities: int, deg: int,
                    intra: int) -> CSR:
    """Community c(v) = floor(communities*v/n).  Each vertex draws ``intra``
    sources uniformly inside its community and ``deg - intra`` uniformly over
    all vertices; duplicates and self-loops kept."""
    v = np.arange(n, dtype=np.int64)
    comm = (communities * v) // n
    # community c spans [lo(c), lo(c+1)) with lo(c) = ceil(c*n/communities)
    lo_all = -((-np.arange(communities + 1, dtype=np.int64) * n) // communities)
    lo = lo_all[comm]
    size = lo_all[comm + 1] - lo
    u = rng.random((n, intra))
    intra_src = lo[:, None] + np.floor(u * size[:, None]).astype(np.int64)
    inter_src = rng.integers(0, n, size=(n, deg - intra), dtype=np.int64)
    src = np.concatenate([intra_src, inter_src], axis=1).astype(np.int32)
    src.sort(axis=1)
    indptr = (np.arange(n + 1, dtype=np.int64) * deg).astype(np.int32)
    return CSR(n, n, indptr, src.reshape(-1), None)


RMAT_ABCD = (0.57, 0.19, 0.19, 0.05)


def _rmat_chunk(seq: np.random.SeedSequence, k: int, scale: int, n: int,
                thresholds, chunk: int):
    """Chunk ``k`` of R-MAT draws, from its own child seed; returns the
    accepted (dst, src) pairs in draw order."""
    rng = np.random.default_rng(
        np.random.SeedSequence(entropy=seq.entropy, spawn_key=tuple(seq.spawn_key) + (k,)))
    t_a, t_ab, t_abc = thresholds
    d_acc = np.zeros(chunk, dtype=np.int32)
    s_acc = np.zeros(chunk, dtype=np.int32)
    for _ in range(scale):
        u = rng.random(chunk, dtype=np.float32)
        rbit = u >= t_ab
        cbit = (u >= t_abc) | ((u >= t_a) & ~rbit)
        d_acc <<= 1
        d_acc |= rbit
        s_acc <<= 1
        s_acc |= cbit
    keep = (d_acc < n) & (s_acc < n) & (d_acc != s_acc)
    return d_acc[keep], s_acc[keep]


def rmat_graph(seq: np.random.SeedSequence, perm_rng: Optional[np.random.Generator],
               scale: int, n: int, e: int, abcd: Sequence[float] = RMAT_ABCD,
               chunk: int = 1 << 24, workers: int = 8) -> CSR:
    """R-MAT edges on a 2^scale grid.

    Each level draws one U[0,1) (float32) and picks a quadrant with
    probabilities (a, b, c, d): the row bit goes to the destination, the
    column bit to the source, most significant bit first.  Draws happen in
    fixed chunks of ``chunk`` edges, chunk k drawing from child seed k of
    ``seq``; an edge is rejected when either end is >= n or when it is a
    self-loop; the accepted edges of chunks 0, 1, ... are concatenated and cut
    at exactly ``e``.  Both ends are then relabelled by one seeded permutation
    of [0, n) (skipped when ``perm_rng`` is None).  Duplicates are kept.
    """
    from concurrent.futures import ThreadPoolExecutor

    a, b, c, _ = abcd
    thr = (np.float32(a), np.float32(a + b), np.float32(a + b + c))
    dst_parts, src_parts = [], []
    got = 0
    k = 0
    with ThreadPoolExecutor(max_workers=workers) as ex:
        while got < e:
            # expected acceptance is high; draw a batch of chunks in parallel
            need = max(1, min(workers, -(-(e - got) // chunk) + 1))
            futs = [ex.submit(_rmat_chunk, seq, k + i, scale, n, thr, chunk)
                    for i in range(need)]
            k += need
            for f in futs:
                d_acc, s_acc = f.result()
                if got >= e:
                    continue
                take = min(e - got, d_acc.size)
                dst_parts.append(d_acc[:take])
                src_parts.append(s_acc[:take])
                got += take
    dst = np.concatenate(dst_parts)
    src = np.concatenate(src_parts)
    del dst_parts, src_parts
    if perm_rng is not None:
        perm = perm_rng.permutation(n).astype(np.int32)
        dst = perm[dst]
        src = perm[src]
    return coo_to_csr(dst, src, n, n)


def two_class_graph(rng: np.random.Generator, perm_rng: Optional[np.random.Generator], n: int,
                    n_hot: int, e: int, p_hot: float) -> CSR:
    """Random multigraph with two degree classes: both ends of every edge are
    drawn independently, from the n_hot "hot" vertices with probability p_hot
    (uniformly inside the class) and from the other n - n_hot vertices
    otherwise, so hot vertices average e * p_hot / n_hot in- and out-edges.
    Duplicates and self-loops are kept; labels are then scrambled by a seeded
    permutation of [0, n) (perm_rng None keeps the hot vertices first)."""
    def ends():
        hot = rng.random(e, dtype=np.float32) < np.float32(p_hot)
        ids = rng.integers(0, n - n_hot, e, dtype=np.int64) + n_hot
        ids[hot] = rng.integers(0, n_hot, int(hot.sum()), dtype=np.int64)
        return ids

    src = ends()
    dst = ends()
    if perm_rng is not None:
        perm = perm_rng.permutation(n)
        src, dst = perm[src], perm[dst]
    return coo_to_csr(dst, src, n, n)


def small_random_graph(rng: np.random.Generator, n_rows: int, n_cols: int, e: int,
                       empty_frac: float = 0.0) -> CSR:
    """Uniform random multigraph for pins and edge cases: destinations are
    drawn from the rows not forced empty."""
    live = np.arange(n_rows)
    if empty_frac > 0 and n_rows > 1:
        k = int(round(n_rows * (1.0 - empty_frac)))
        live = rng.choice(n_rows, size=max(k, 1), replace=False)
    dst = live[rng.integers(0, live.size, size=e)]
    src = rng.integers(0, n_cols, size=e)
    return coo_to_csr(dst, src, n_rows, n_cols)


# --------------------------------------------------------------------------
# the five benchmark / parity workloads
# --------------------------------------------------------------------------

CONFIG_NAMES = (
    "tiny_uniform_1k",      # N=1,024, E=16,384, d=32
    "uniform_deg100_100k",  # N=100,000, in-degree 100, d in {32..512}
    "rmat_233k_115m",       # R-MAT N=232,965, E=114.6M, d=128
    "clustered_133k_deg300",  # N=132,534, 100 communities, deg 300, H=8 x 16
    "rmat_1m_33m_train",    # R-MAT N=2^20, E=2^25, d=256, CSR + CSC
    "rand_100k_48m",        # two degree classes: 20K at ~2000, 80K at ~100, E=48M, d in {32..512}
)

_SEEDS = {name: i + 1 for i, name in enumerate(CONFIG_NAMES)}


def _children(seed: int, k: int):
    return np.random.SeedSequence(seed).spawn(k)


def make_config(name: str, d: Optional[int] = None, scale_down: int = 1) -> Workload:
    """Build one of the named workloads.

    ``scale_down`` > 1 shrinks vertex and edge counts of the two R-MAT
    workloads and the clustered one (for quick parity runs) while keeping the
    generator, its parameters and the degree structure family.
    """
    if name not in _SEEDS:
        raise KeyError(name)
    seed = _SEEDS[name]
    s_struct, s_feat, s_edge, s_grad, s_perm = _children(seed, 5)
    r_struct, r_feat, r_edge, r_grad, r_perm = (
        np.random.default_rng(s) for s in (s_struct, s_feat, s_edge, s_grad, s_perm))
    arrays: Dict[str, np.ndarray] = {}
    meta: Dict[str, object] = {"seed": seed, "scale_down": scale_down}
    csc = None
    if name == "tiny_uniform_1k":
        csr = uniform_graph(r_struct, 1024, 16384)
        arrays["x"] = r_feat.uniform(-1.0, 1.0, size=(1024, 32)).astype(np.float32)
        meta.update(heads=1, head_dim=32)
    elif name == "uniform_deg100_100k":
        d = 128 if d is None else d
        n = 100_000 // scale_down
        csr = fixed_indegree_graph(r_struct, n, 100)
        # a separate feature stream per width
        r_d = np.random.default_rng(np.random.SeedSequence([seed, d]))
        arrays["x"] = r_d.standard_normal((n, d), dtype=np.float32)
        meta.update(heads=1, head_dim=d)
    elif name == "rmat_233k_115m":
        d = 128 if d is None else d
        n = 232_965 // scale_down
        e = 114_600_000 // scale_down
        scale = int(np.ceil(np.log2(n)))
        csr = rmat_graph(s_struct, r_perm, scale, n, e)
        arrays["x"] = r_feat.standard_normal((n, d), dtype=np.float32)
        arrays["w"] = (np.float32(1.0) - r_edge.random(csr.nnz, dtype=np.float32))
        meta.update(heads=1, head_dim=d, rmat_scale=scale)
    elif name == "clustered_133k_deg300":
        n = 132_534 // scale_down
        csr = clustered_graph(r_struct, n, 100, 300, 270)
        arrays["x"] = r_feat.standard_normal((n, 8, 16), dtype=np.float32)
        meta.update(heads=8, head_dim=16)
    elif name == "rand_100k_48m":
        d = 128 if d is None else d
        n = 100_000 // scale_down
        csr = two_class_graph(r_struct, r_perm, n, n // 5, 48_000_000 // scale_down, 40.0 / 48.0)
        r_d = np.random.default_rng(np.random.SeedSequence([seed, d]))
        arrays["x"] = r_d.standard_normal((n, d), dtype=np.float32)
        meta.update(heads=1, head_dim=d)
    else:  # rmat_1m_33m_train
        d = 256 if d is None else d
        n = (1 << 20) // scale_down
        e = (1 << 25) // scale_down
        scale = int(np.ceil(np.log2(n)))
        csr = rmat_graph(s_struct, r_perm, scale, n, e)
        csc = csr_to_csc(csr)
        arrays["x"] = r_feat.standard_normal((n, d), dtype=np.float32)
        arrays["dy"] = r_grad.standard_normal((n, d), dtype=np.float32)
        meta.update(heads=1, head_dim=d, rmat_scale=scale)
    meta["num_rows"] = csr.num_rows
    meta["nnz"] = csr.nnz
    return Workload(name, csr, csc, arrays, meta)
