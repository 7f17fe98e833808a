"""ctypes shim for the C oracle in ``fgref.c`` (test infrastructure only).

``build()`` compiles the oracle with gcc (no -march=native, so the library runs
on any x86-64 host; -ffp-contract=off so the C source's roundings are the ones
that happen).  The wrappers take numpy arrays and a ``synth.CSR``-like object
(``num_rows``, ``num_cols``, ``indptr``, ``indices``, ``edge_ids``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fgref.c")
# FGREF_LIB points the shim at another build of the oracle (the mutation test
# plants mistakes in copies of fgref.c and checks that the pins catch them)
_LIB = os.environ.get("FGREF_LIB") or os.path.join(_HERE, "_build", "libfgref.so")

MSG_COPY_SRC, MSG_SRC_MUL_EDGE = 0, 1
RED_SUM, RED_MAX = 0, 1

_lib = None


def lib_path() -> str:
    return _LIB


# Portable flags (no -march=native): the library is built once and may run
# on a host with another CPU model.
BUILD_FLAGS = ["-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math"]


def compile_oracle(src: str, out: str) -> str:
    """gcc build of an oracle source file into a shared library."""
    os.makedirs(os.path.dirname(out), exist_ok=True)
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc"] + BUILD_FLAGS + ["-fPIC", "-shared", "-Wall", "-Wextra",
                                   "-Wno-unused-parameter", "-o", tmp, src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build(force: bool = True) -> str:
    """Compile the oracle library; returns its path."""
    if not force and os.path.exists(_LIB):
        return _LIB
    return compile_oracle(_SRC, _LIB)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    i64, i32p = ctypes.c_int64, ctypes.c_void_p
    vp = ctypes.c_void_p
    lib.fgref_gspmm.argtypes = [i64, i64, vp, vp, vp, i64, ctypes.c_int, ctypes.c_int, i64, i64,
                                vp, vp, vp, i64, vp, vp, vp, ctypes.c_int]
    lib.fgref_gsddmm.argtypes = [i64, i64, vp, vp, vp, i64, i64, i64, vp, vp, vp, i64, vp, vp,
                                 ctypes.c_int]
    lib.fgref_edge_softmax.argtypes = [i64, vp, vp, i64, i64, vp, ctypes.c_int, ctypes.c_float,
                                       vp, i64, vp, ctypes.c_int]
    lib.fgref_gspmm_max_backward.argtypes = [i64, i64, vp, vp, vp, i64, ctypes.c_int, i64, i64,
                                             vp, vp, vp, vp, i64, vp, vp, vp, vp, ctypes.c_int]
    lib.fgref_edge_softmax_backward.argtypes = [i64, vp, vp, i64, i64, vp, vp, ctypes.c_int,
                                                ctypes.c_float, vp, i64, vp, vp, ctypes.c_int]
    for f in (lib.fgref_gspmm, lib.fgref_gsddmm, lib.fgref_edge_softmax,
              lib.fgref_gspmm_max_backward, lib.fgref_edge_softmax_backward):
        f.restype = ctypes.c_int
    lib.fgref_max_threads.restype = ctypes.c_int
    lib.fgref_mlp_aggregate.argtypes = [i64, i64, vp, vp, vp, i64, i64, i64, vp, vp, vp, vp, i64,
                                        vp, vp, vp, ctypes.c_int]
    lib.fgref_mlp_aggregate.restype = ctypes.c_int
    lib.fgref_dense_matmul.argtypes = [i64, i64, i64, vp, vp, vp, ctypes.c_int]
    lib.fgref_dense_matmul.restype = ctypes.c_int
    lib.fgref_set_num_threads.argtypes = [ctypes.c_int]
    lib.fgref_set_num_threads.restype = None
    del i32p
    _lib = lib
    return lib


def max_threads() -> int:
    return int(_load().fgref_max_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads for later calls made with threads=0."""
    _load().fgref_set_num_threads(int(n))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    if a is None:
        return None
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _graph_args(g):
    indptr = _c(g.indptr, np.int32)
    indices = _c(g.indices, np.int32)
    eids = _c(g.edge_ids, np.int32) if getattr(g, "edge_ids", None) is not None else None
    return indptr, indices, eids


def _rows_arg(rows, num_rows):
    if rows is None:
        return None, num_rows
    r = np.ascontiguousarray(rows, dtype=np.int64)
    return r, r.size


def gspmm(g, x: np.ndarray, msg: int = MSG_COPY_SRC, red: int = RED_SUM, heads: int = 1,
          edge_val: Optional[np.ndarray] = None, rows: Optional[Sequence[int]] = None,
          nnz_total: Optional[int] = None, with_norm: bool = False, threads: int = 0):
    """Returns out [sel, F] (and arg for max, and term norms if asked)."""
    lib = _load()
    indptr, indices, eids = _graph_args(g)
    x = _c(x, np.float32).reshape(g.num_cols, -1)
    F = x.shape[1]
    if F % heads:
        raise ValueError("feature width not divisible by heads")
    dh = F // heads
    ev = _c(edge_val, np.float32)
    r, nsel = _rows_arg(rows, g.num_rows)
    out = np.empty((nsel, F), np.float32)
    arg = np.empty((nsel, F), np.int32) if red == RED_MAX else None
    norm = np.empty((nsel, F), np.float64) if with_norm else None
    nt = int(indptr[-1]) if nnz_total is None else nnz_total
    rc = lib.fgref_gspmm(g.num_rows, g.num_cols, _ptr(indptr), _ptr(indices), _ptr(eids), nt,
                         msg, red, heads, dh, _ptr(x), _ptr(ev), _ptr(r), nsel, _ptr(out),
                         _ptr(arg), _ptr(norm), threads)
    if rc != 0:
        raise ValueError("fgref_gspmm failed (%d)" % rc)
    res = [out]
    if red == RED_MAX:
        res.append(arg)
    if with_norm:
        res.append(norm)
    return res[0] if len(res) == 1 else tuple(res)


def gsddmm(g, xs: np.ndarray, xd: np.ndarray, heads: int = 1,
           rows: Optional[Sequence[int]] = None, nnz_total: Optional[int] = None,
           out: Optional[np.ndarray] = None, with_norm: bool = False, threads: int = 0):
    """Returns out [nnz_total, H] indexed by edge id (and term norms)."""
    lib = _load()
    indptr, indices, eids = _graph_args(g)
    xs = _c(xs, np.float32).reshape(g.num_cols, -1)
    xd = _c(xd, np.float32).reshape(g.num_rows, -1)
    F = xs.shape[1]
    if xd.shape[1] != F or F % heads:
        raise ValueError("bad feature widths")
    dh = F // heads
    nt = int(indptr[-1]) if nnz_total is None else nnz_total
    if out is None:
        out = np.full((nt, heads), np.nan, np.float32)
    norm = np.full((nt, heads), np.nan, np.float64) if with_norm else None
    r, nsel = _rows_arg(rows, g.num_rows)
    rc = lib.fgref_gsddmm(g.num_rows, g.num_cols, _ptr(indptr), _ptr(indices), _ptr(eids), nt,
                          heads, dh, _ptr(xs), _ptr(xd), _ptr(r), nsel, _ptr(out), _ptr(norm),
                          threads)
    if rc != 0:
        raise ValueError("fgref_gsddmm failed (%d)" % rc)
    return (out, norm) if with_norm else out


def edge_softmax(g, scores: np.ndarray, heads: int = 1, leaky: bool = True,
                 slope: float = 0.2, rows: Optional[Sequence[int]] = None,
                 nnz_total: Optional[int] = None, out: Optional[np.ndarray] = None,
                 threads: int = 0):
    """Returns out [nnz_total, H] indexed by edge id."""
    lib = _load()
    indptr, _, eids = _graph_args(g)
    nt = int(indptr[-1]) if nnz_total is None else nnz_total
    s = _c(scores, np.float32).reshape(nt, heads)
    if out is None:
        out = np.full((nt, heads), np.nan, np.float32)
    r, nsel = _rows_arg(rows, g.num_rows)
    rc = lib.fgref_edge_softmax(g.num_rows, _ptr(indptr), _ptr(eids), nt, heads, _ptr(s),
                                int(bool(leaky)), float(slope), _ptr(r), nsel, _ptr(out),
                                threads)
    if rc != 0:
        raise ValueError("fgref_edge_softmax failed (%d)" % rc)
    return out


def gspmm_max_backward(g, x: np.ndarray, grad_out: np.ndarray, msg: int = MSG_COPY_SRC,
                       heads: int = 1, edge_val: Optional[np.ndarray] = None,
                       rows: Optional[Sequence[int]] = None, nnz_total: Optional[int] = None,
                       want_edge: bool = False, with_norm: bool = False, threads: int = 0):
    """Gradient of gSpMM-max w.r.t. the source features (and the edge values
    for src_mul_edge when want_edge): returns grad_src [num_cols, F]
    (, grad_edge [nnz_total, H]) (, src_norm (, edge_norm))."""
    lib = _load()
    indptr, indices, eids = _graph_args(g)
    x = _c(x, np.float32).reshape(g.num_cols, -1)
    F = x.shape[1]
    if F % heads:
        raise ValueError("feature width not divisible by heads")
    dh = F // heads
    go = _c(grad_out, np.float32).reshape(g.num_rows, F)
    ev = _c(edge_val, np.float32)
    nt = int(indptr[-1]) if nnz_total is None else nnz_total
    r, nsel = _rows_arg(rows, g.num_rows)
    gsrc = np.empty((g.num_cols, F), np.float32)
    gedge = np.empty((nt, heads), np.float32) if want_edge else None
    snorm = np.empty((g.num_cols, F), np.float64) if with_norm else None
    enorm = np.empty((nt, heads), np.float64) if (with_norm and want_edge) else None
    rc = lib.fgref_gspmm_max_backward(g.num_rows, g.num_cols, _ptr(indptr), _ptr(indices),
                                      _ptr(eids), nt, msg, heads, dh, _ptr(x), _ptr(ev), _ptr(go),
                                      _ptr(r), nsel, _ptr(gsrc), _ptr(gedge), _ptr(snorm),
                                      _ptr(enorm), threads)
    if rc != 0:
        raise ValueError("fgref_gspmm_max_backward failed (%d)" % rc)
    res = [gsrc]
    if want_edge:
        res.append(gedge)
    if with_norm:
        res.append(snorm)
        if want_edge:
            res.append(enorm)
    return res[0] if len(res) == 1 else tuple(res)


def edge_softmax_backward(g, scores: np.ndarray, grad_out: np.ndarray, heads: int = 1,
                          leaky: bool = True, slope: float = 0.2,
                          rows: Optional[Sequence[int]] = None, nnz_total: Optional[int] = None,
                          out: Optional[np.ndarray] = None, with_scale: bool = False,
                          threads: int = 0):
    """Gradient of edge softmax w.r.t. the scores: [nnz_total, H] by edge id
    (edges of unselected rows untouched) (, term scale)."""
    lib = _load()
    indptr, _, eids = _graph_args(g)
    nt = int(indptr[-1]) if nnz_total is None else nnz_total
    s = _c(scores, np.float32).reshape(nt, heads)
    go = _c(grad_out, np.float32).reshape(nt, heads)
    if out is None:
        out = np.full((nt, heads), np.nan, np.float32)
    sc = np.full((nt, heads), np.nan, np.float64) if with_scale else None
    r, nsel = _rows_arg(rows, g.num_rows)
    rc = lib.fgref_edge_softmax_backward(g.num_rows, _ptr(indptr), _ptr(eids), nt, heads, _ptr(s),
                                         _ptr(go), int(bool(leaky)), float(slope), _ptr(r), nsel,
                                         _ptr(out), _ptr(sc), threads)
    if rc != 0:
        raise ValueError("fgref_edge_softmax_backward failed (%d)" % rc)
    return (out, sc) if with_scale else out


def mlp_aggregate(g, xs: np.ndarray, xd: np.ndarray, w: np.ndarray,
                  rows: Optional[Sequence[int]] = None, nnz_total: Optional[int] = None,
                  with_scale: bool = False, threads: int = 0):
    """MLP aggregation: returns out [sel, d_out], arg [sel, d_out] (, scale)."""
    lib = _load()
    indptr, indices, eids = _graph_args(g)
    w = _c(w, np.float32)
    d_in, d_out = w.shape
    xs = _c(xs, np.float32).reshape(g.num_cols, d_in)
    xd = _c(xd, np.float32).reshape(g.num_rows, d_in)
    nt = int(indptr[-1]) if nnz_total is None else nnz_total
    r, nsel = _rows_arg(rows, g.num_rows)
    out = np.empty((nsel, d_out), np.float32)
    arg = np.empty((nsel, d_out), np.int32)
    sc = np.empty((nsel, d_out), np.float64) if with_scale else None
    rc = lib.fgref_mlp_aggregate(g.num_rows, g.num_cols, _ptr(indptr), _ptr(indices), _ptr(eids),
                                 nt, d_in, d_out, _ptr(xs), _ptr(xd), _ptr(w), _ptr(r), nsel,
                                 _ptr(out), _ptr(arg), _ptr(sc), threads)
    if rc != 0:
        raise ValueError("fgref_mlp_aggregate failed (%d)" % rc)
    return (out, arg, sc) if with_scale else (out, arg)


def dense_matmul(x: np.ndarray, w: np.ndarray, threads: int = 0) -> np.ndarray:
    """Y = X W, the dense vertex transform of MLP aggregation (Fig. 3b's
    vector-matrix product applied per vertex): fp32 inputs, fp64 products,
    sums and result (fgref_dense_matmul)."""
    lib = _load()
    w = _c(w, np.float32)
    if w.ndim != 2:
        raise ValueError("w must be [d_in, d_out]")
    d_in, d_out = w.shape
    x = _c(x, np.float32).reshape(-1, d_in)
    y = np.empty((x.shape[0], d_out), np.float64)
    rc = lib.fgref_dense_matmul(x.shape[0], d_in, d_out, _ptr(x), _ptr(w), _ptr(y), threads)
    if rc != 0:
        raise ValueError("fgref_dense_matmul failed (%d)" % rc)
    return y
