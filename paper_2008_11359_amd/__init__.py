"""gfx950 (MI355X) generalized SpMM / SDDMM / edge softmax -- Python binding.

Thin ctypes marshalling over the C ABI declared in ``include/featgraph_hip.h``
(library ``_build/libfeatgraph_hip.so``).  PyTorch provides device memory and
the current HIP stream; every step of the computation runs in the library's
kernels.  There is no CPU fallback: importing this package fails when the
library has not been built, and calls fail when a tensor is not on the GPU.

    g = Graph.from_csr(csr)                   # device copy of a CSR (rows = destinations)
    plan = Plan(g, max_width=128)             # degree-aware schedule, built once per graph
    h = gspmm(g, x, plan=plan)                # copy_src + sum      (GCN aggregation, Eq. 3)
    h, arg = gspmm(g, x, reduce="max", plan=plan)
    s = gsddmm(g, x, x, plan=plan)            # per-edge dot        (Eq. 4)
    a = edge_softmax(g, s, leaky=True, slope=0.2, plan=plan)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

try:
    import torch
except ImportError as exc:  # pragma: no cover
    raise ImportError("paper_2008_11359_amd needs PyTorch (ROCm) for device memory") from exc

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_build", "libfeatgraph_hip.so")

FG_OK, FG_ERR_INVALID_ARG, FG_ERR_UNSUPPORTED, FG_ERR_HIP, FG_ERR_NO_MEMORY = 0, -1, -2, -3, -4
FG_ERR_SCRATCH_LIMIT = -5
NOALLOC_SCRATCH_BYTES = 32 << 20  # fixed scratch of gspmm_noalloc (per device)
MSG_OPS = {"copy_src": 0, "src_mul_edge": 1}
REDUCE_OPS = {"sum": 0, "max": 1}
EDGE_OPS = {"dot": 0}
ABI_VERSION = 4


class FgError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__("%s: %s (status %d)" % (what, status_string(status), status))
        self.status = status


class _Graph(ctypes.Structure):
    _fields_ = [
        ("num_rows", ctypes.c_int64),
        ("num_cols", ctypes.c_int64),
        ("nnz", ctypes.c_int64),
        ("nnz_total", ctypes.c_int64),
        ("indptr", ctypes.c_void_p),
        ("indices", ctypes.c_void_p),
        ("edge_ids", ctypes.c_void_p),
    ]


class _PlanOptions(ctypes.Structure):
    _fields_ = [("segment_edges", ctypes.c_int32), ("max_row_segments", ctypes.c_int32),
                ("source_slab_rows", ctypes.c_int32), ("partition_min_degree", ctypes.c_int32),
                ("item_order", ctypes.c_int32), ("max_backward", ctypes.c_int32),
                ("softmax_segment_edges", ctypes.c_int32), ("band_row_edges", ctypes.c_int32),
                ("reserved", ctypes.c_int32 * 2)]


class _PlanInfo(ctypes.Structure):
    _fields_ = [
        ("num_rows", ctypes.c_int64),
        ("nnz", ctypes.c_int64),
        ("num_segments", ctypes.c_int64),
        ("num_split_rows", ctypes.c_int64),
        ("num_slots", ctypes.c_int64),
        ("num_partitioned_rows", ctypes.c_int64),
        ("plain_segments", ctypes.c_int64),
        ("plain_split_rows", ctypes.c_int64),
        ("plain_slots", ctypes.c_int64),
        ("max_width", ctypes.c_int64),
        ("workspace_bytes", ctypes.c_int64),
        ("segment_edges", ctypes.c_int32),
        ("max_row_segments", ctypes.c_int32),
        ("source_slab_rows", ctypes.c_int32),
        ("partition_min_degree", ctypes.c_int32),
        ("item_order", ctypes.c_int32),
        ("max_backward", ctypes.c_int32),
        ("indptr_checksum", ctypes.c_uint64),
        ("sddmm_segments", ctypes.c_int64),
    ]


class Segment(ctypes.Structure):
    _fields_ = [("row", ctypes.c_int32), ("begin", ctypes.c_int32), ("end", ctypes.c_int32),
                ("slot", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            "HIP library %s is missing: build it with `python paper_2008_11359_amd/build.py` "
            "(there is no CPU fallback)" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    gp = ctypes.POINTER(_Graph)
    lib.fg_status_string.restype = ctypes.c_char_p
    lib.fg_status_string.argtypes = [ctypes.c_int]
    lib.fg_abi_version.restype = i32
    lib.fg_schedule_host.restype = ctypes.c_int
    lib.fg_schedule_host.argtypes = [vp, vp, i64, i64, i64, ctypes.POINTER(_PlanOptions), i32,
                                     vp, i64, ctypes.POINTER(i64), ctypes.POINTER(i64),
                                     ctypes.POINTER(i64)]
    lib.fg_plan_create.restype = ctypes.c_int
    lib.fg_plan_create.argtypes = [gp, vp, vp, i64, ctypes.POINTER(_PlanOptions),
                                   ctypes.POINTER(vp), vp]
    lib.fg_plan_destroy.restype = ctypes.c_int
    lib.fg_plan_destroy.argtypes = [vp]
    lib.fg_plan_get_info.restype = ctypes.c_int
    lib.fg_plan_get_info.argtypes = [vp, ctypes.POINTER(_PlanInfo)]
    lib.fg_indptr_checksum.restype = ctypes.c_int
    lib.fg_indptr_checksum.argtypes = [vp, i64, ctypes.POINTER(ctypes.c_uint64)]
    lib.fg_plan_validate.restype = ctypes.c_int
    lib.fg_plan_validate.argtypes = [vp, gp, vp, vp]
    lib.fg_gspmm.restype = ctypes.c_int
    lib.fg_gspmm.argtypes = [gp, ctypes.c_int, ctypes.c_int, i32, i64, vp, vp, vp, vp, vp, vp]
    lib.fg_gspmm_noalloc.restype = ctypes.c_int
    lib.fg_gspmm_noalloc.argtypes = [gp, ctypes.c_int, ctypes.c_int, i32, i64, vp, vp, vp, vp, vp,
                                     vp]
    lib.fg_gsddmm.restype = ctypes.c_int
    lib.fg_gsddmm.argtypes = [gp, ctypes.c_int, i32, i64, vp, vp, vp, vp, vp]
    lib.fg_gat_aggregate.restype = ctypes.c_int
    lib.fg_gat_aggregate.argtypes = [gp, i32, i64, vp, vp, i32, ctypes.c_float, vp, vp, vp]
    lib.fg_edge_softmax.restype = ctypes.c_int
    lib.fg_edge_softmax.argtypes = [gp, i32, vp, i32, ctypes.c_float, vp, vp, vp]
    lib.fg_gspmm_max_backward.restype = ctypes.c_int
    lib.fg_gspmm_max_backward.argtypes = [gp, ctypes.c_int, i32, i64, vp, vp, vp, vp, vp, vp, vp,
                                          vp]
    lib.fg_edge_softmax_backward.restype = ctypes.c_int
    lib.fg_edge_softmax_backward.argtypes = [gp, i32, vp, vp, vp, i32, ctypes.c_float, vp, vp, vp]
    lib.fg_gsddmm_edge_softmax_backward.restype = ctypes.c_int
    lib.fg_gsddmm_edge_softmax_backward.argtypes = [gp, i32, i64, vp, vp, vp, vp, i32,
                                                    ctypes.c_float, vp, vp, vp]
    lib.fg_gsddmm_edge_softmax.restype = ctypes.c_int
    lib.fg_gsddmm_edge_softmax.argtypes = [gp, i32, i64, vp, vp, i32, ctypes.c_float, vp, vp, vp,
                                           vp]
    lib.fg_dense_matmul.restype = ctypes.c_int
    lib.fg_dense_matmul.argtypes = [i64, i64, i64, vp, vp, vp, vp]
    lib.fg_mlp_aggregate.restype = ctypes.c_int
    lib.fg_mlp_aggregate.argtypes = [gp, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp]
    if lib.fg_abi_version() != ABI_VERSION:
        raise ImportError("ABI version mismatch: library %d, binding %d"
                          % (lib.fg_abi_version(), ABI_VERSION))
    return lib


_lib = _load()


def status_string(status: int) -> str:
    return _lib.fg_status_string(int(status)).decode()


def _check(status: int, what: str) -> None:
    if status != FG_OK:
        raise FgError(status, what)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _dev_tensor(t: torch.Tensor, dtype: torch.dtype, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor (there is no CPU path)" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


# ----------------------------------------------------------------------------
# graphs and plans
# ----------------------------------------------------------------------------


class Graph:
    """A CSR graph in device memory; rows are destination vertices.

    ``edge_ids`` (optional) gives each stored edge's id; ``nnz_total`` is the
    size of the edge-id space (for a transposed graph: the CSR's nnz).
    """

    def __init__(self, num_rows: int, num_cols: int, indptr: torch.Tensor, indices: torch.Tensor,
                 edge_ids: Optional[torch.Tensor] = None, nnz_total: int = 0,
                 indptr_host: Optional[np.ndarray] = None,
                 indices_host: Optional[np.ndarray] = None):
        self.indptr = _dev_tensor(indptr, torch.int32, "indptr")
        self.indices = _dev_tensor(indices, torch.int32, "indices")
        self.edge_ids = None if edge_ids is None else _dev_tensor(edge_ids, torch.int32, "edge_ids")
        if self.indptr.numel() != num_rows + 1:
            raise ValueError("indptr must have num_rows + 1 entries")
        self.num_rows = int(num_rows)
        self.num_cols = int(num_cols)
        self.nnz = int(self.indices.numel())
        self.nnz_total = int(nnz_total) if nnz_total else self.nnz
        if self.edge_ids is not None and self.edge_ids.numel() != self.nnz:
            raise ValueError("edge_ids must have nnz entries")
        self.indptr_host = None if indptr_host is None else np.ascontiguousarray(
            indptr_host, dtype=np.int32)
        self.indices_host = None if indices_host is None else np.ascontiguousarray(
            indices_host, dtype=np.int32)
        self._c = _Graph(self.num_rows, self.num_cols, self.nnz, self.nnz_total,
                         self.indptr.data_ptr(), self.indices.data_ptr() if self.nnz else None,
                         _ptr(self.edge_ids))

    @classmethod
    def from_csr(cls, csr, device="cuda", nnz_total: int = 0, check: bool = True) -> "Graph":
        """Copies a host CSR (numpy int32 ``indptr``/``indices``/``edge_ids``)
        to the device.  With ``check`` the structure is validated on the host
        first, since the kernels do not range-check indices."""
        indptr = np.ascontiguousarray(csr.indptr, dtype=np.int32)
        indices = np.ascontiguousarray(csr.indices, dtype=np.int32)
        eids = getattr(csr, "edge_ids", None)
        nt = int(nnz_total) if nnz_total else int(indptr[-1])
        if check:
            _check_host_csr(csr.num_rows, csr.num_cols, indptr, indices, eids, nt)
        dev = torch.device(device)
        t_ip = torch.from_numpy(indptr).to(dev)
        t_ix = torch.from_numpy(indices).to(dev)
        t_e = None if eids is None else torch.from_numpy(
            np.ascontiguousarray(eids, dtype=np.int32)).to(dev)
        return cls(csr.num_rows, csr.num_cols, t_ip, t_ix, t_e, nt, indptr_host=indptr,
                   indices_host=indices)


def _check_host_csr(num_rows, num_cols, indptr, indices, eids, nnz_total):
    if indptr.shape != (num_rows + 1,) or indptr[0] != 0:
        raise ValueError("bad indptr")
    if num_rows and np.any(np.diff(indptr.astype(np.int64)) < 0):
        raise ValueError("indptr must be nondecreasing")
    nnz = int(indptr[-1])
    if indices.shape != (nnz,):
        raise ValueError("indices must have indptr[-1] entries")
    if nnz and (indices.min() < 0 or indices.max() >= num_cols):
        raise ValueError("indices out of range")
    if eids is not None:
        eids = np.asarray(eids)
        if eids.shape != (nnz,) or (nnz and (eids.min() < 0 or eids.max() >= nnz_total)):
            raise ValueError("edge_ids out of range")
    elif nnz_total < nnz:
        raise ValueError("nnz_total smaller than nnz")


class Plan:
    """Degree-aware schedules of one graph (see fg_plan_create): rows longer
    than ``segment_edges`` (default 1536 edges in the gather schedule of
    gSpMM / gSDDMM, 16,384 in the edge-softmax schedule, which
    ``softmax_segment_edges`` sets apart) are cut into equal pieces (at most
    ``max_row_segments``); long rows of the gather schedule may also be cut
    at source-slab boundaries, so that each die gathers from a narrow band of
    the features.  ``source_slab_rows``: 0 (default) automatic slabs once the
    num_cols x max_width features exceed 128 MiB, or 32 MiB when the gathers
    are spread (no dominant hot sources, no locality along row ids); -1 once
    they exceed 32 MiB; -2 never; > 0 that many source ids per slab.  ``item_order``: 1 longest
    item first, 2 by power-of-two length class with rows in id order (keeps
    the locality of graphs whose neighbouring ids share sources), 3 the items
    of 1 with rows of more than ``band_row_edges`` edges (default 256; -1:
    none) cut into at least 8 pieces and the pieces of split rows dealt to
    the dies by position in the row (each die gathers from about one eighth
    of their sources; with ``band_row_edges=-1`` the results equal those of
    1), 0 (default) picks 2 for such graphs and otherwise 3 if some row is
    cut into 8 or more pieces by length, else 1.  Partial-result
    workspace for features up to ``max_width`` floats.  ``max_backward``:
    also hold the workspace with which gspmm_max_backward bins the gradient
    per source tile instead of adding it with atomics (8 bytes per element of
    a num_rows x max_width gradient).  Zero selects the library defaults.
    Owns device memory until ``close()``."""

    def __init__(self, g: Graph, max_width: int, segment_edges: int = 0,
                 max_row_segments: int = 0, source_slab_rows: int = 0,
                 partition_min_degree: int = 0, item_order: int = 0,
                 max_backward: bool = False, softmax_segment_edges: int = 0,
                 band_row_edges: int = 0):
        opt = _options(segment_edges, max_row_segments, source_slab_rows, partition_min_degree,
                       item_order, max_backward, softmax_segment_edges, band_row_edges)
        h = ctypes.c_void_p()
        ip, ix = g.indptr_host, g.indices_host
        st = _lib.fg_plan_create(ctypes.byref(g._c), None if ip is None else ip.ctypes.data,
                                 None if ix is None else ix.ctypes.data, int(max_width),
                                 ctypes.byref(opt), ctypes.byref(h), _stream())
        _check(st, "fg_plan_create")
        self._h = h
        self.graph = g
        self._versions = _graph_versions(g)

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("plan is closed")
        return self._h

    def validate(self) -> None:
        """Re-checks the plan against its graph's current indptr on the device
        (fg_plan_validate: the checksum taken at creation); raises FgError if
        indptr no longer matches.  Afterwards in-place edits that kept indptr
        (and a re-sorted indices of an unpartitioned plan) are accepted."""
        g = self.graph
        _check(_lib.fg_plan_validate(self.handle, ctypes.byref(g._c), None, _stream()),
               "fg_plan_validate")
        self._versions = _graph_versions(g)

    def check_current(self) -> None:
        """Raises ValueError when the graph's device arrays were modified in
        place since the plan was built (or last validated): the plan's
        schedules describe the old rows."""
        if _graph_versions(self.graph) != self._versions:
            raise ValueError(
                "the graph's indptr / indices / edge_ids were modified in place after this plan "
                "was built; build a new plan, or call plan.validate() if indptr is unchanged")

    def info(self) -> dict:
        inf = _PlanInfo()
        _check(_lib.fg_plan_get_info(self.handle, ctypes.byref(inf)), "fg_plan_get_info")
        return {k: getattr(inf, k) for k, _ in _PlanInfo._fields_}

    def close(self) -> None:
        if self._h is not None:
            torch.cuda.current_stream().synchronize()
            _check(_lib.fg_plan_destroy(self._h), "fg_plan_destroy")
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _options(segment_edges: int = 0, max_row_segments: int = 0, source_slab_rows: int = 0,
             partition_min_degree: int = 0, item_order: int = 0,
             max_backward: bool = False, softmax_segment_edges: int = 0,
             band_row_edges: int = 0) -> _PlanOptions:
    opt = _PlanOptions()
    opt.segment_edges = int(segment_edges)
    opt.max_row_segments = int(max_row_segments)
    opt.source_slab_rows = int(source_slab_rows)
    opt.partition_min_degree = int(partition_min_degree)
    opt.item_order = int(item_order)
    opt.max_backward = int(max_backward)
    opt.softmax_segment_edges = int(softmax_segment_edges)
    opt.band_row_edges = int(band_row_edges)
    return opt


def schedule_host(indptr: np.ndarray, indices: Optional[np.ndarray] = None, num_cols: int = 0,
                  max_width: int = 128, which: str = "gather", **options):
    """A plan's schedule computed on the host (no GPU needed); ``indices``
    (with ``num_cols``) enables source partitioning.  Returns (items as an
    [n, 4] int32 array of row, begin, end, slot; num_split_rows, num_slots)."""
    ip = np.ascontiguousarray(indptr, dtype=np.int32)
    ix = None if indices is None else np.ascontiguousarray(indices, dtype=np.int32)
    opt = _options(**options)
    w = {"gather": 0, "plain": 1, "sddmm": 2}[which]
    args = (ip.ctypes.data, None if ix is None else ix.ctypes.data, ip.size - 1, int(num_cols),
            int(max_width), ctypes.byref(opt), w)
    n_seg, n_split, n_slot = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.fg_schedule_host(*args, None, 0, ctypes.byref(n_seg), ctypes.byref(n_split),
                                 ctypes.byref(n_slot)), "fg_schedule_host")
    segs = np.zeros((n_seg.value, 4), np.int32)
    _check(_lib.fg_schedule_host(*args, segs.ctypes.data, n_seg.value, None, None, None),
           "fg_schedule_host")
    return segs, n_split.value, n_slot.value


def _graph_versions(g: Graph):
    """In-place modification counters of a graph's device arrays."""
    return tuple(None if t is None else t._version for t in (g.indptr, g.indices, g.edge_ids))


def indptr_checksum(indptr: np.ndarray) -> int:
    """fg_indptr_checksum of a host indptr (64-bit FNV-1a over its int32 bytes)."""
    ip = np.ascontiguousarray(indptr, dtype=np.int32)
    if ip.ndim != 1 or ip.size < 1:
        raise ValueError("indptr must be a non-empty 1-D array")
    out = ctypes.c_uint64()
    _check(_lib.fg_indptr_checksum(ip.ctypes.data, ip.size - 1, ctypes.byref(out)),
           "fg_indptr_checksum")
    return out.value


def _plan_handle(plan: Optional[Plan]):
    if plan is None:
        return None
    plan.check_current()
    return plan.handle


# ----------------------------------------------------------------------------
# the three operators
# ----------------------------------------------------------------------------


def gspmm(g: Graph, x: torch.Tensor, edge: Optional[torch.Tensor] = None, msg: str = "copy_src",
          reduce: str = "sum", heads: int = 1, plan: Optional[Plan] = None,
          out: Optional[torch.Tensor] = None, arg: Optional[torch.Tensor] = None):
    """Generalized SpMM: out[v] = reduce over in-edges (u -> v, id e) of
    msg(x[u], edge[e]).  x: [num_cols, F] or [num_cols, H, dh] fp32.  edge:
    [nnz_total] or [nnz_total, H] fp32 for msg='src_mul_edge'.  Returns out
    (shape of x with num_rows rows) and, for reduce='max', the int32 edge id
    of each maximum (-1 for rows without edges)."""
    if msg not in MSG_OPS or reduce not in REDUCE_OPS:
        raise ValueError("unknown msg %r or reduce %r" % (msg, reduce))
    x = _dev_tensor(x, torch.float32, "x")
    if x.shape[0] != g.num_cols:
        raise ValueError("x must have num_cols rows")
    F = int(np.prod(x.shape[1:])) if x.dim() > 1 else 1
    if x.dim() == 3:
        heads = int(x.shape[1])
    if F % heads:
        raise ValueError("feature width not divisible by heads")
    dh = F // heads
    if msg == "src_mul_edge":
        if edge is None:
            raise ValueError("src_mul_edge needs edge values")
        edge = _dev_tensor(edge, torch.float32, "edge")
        if edge.numel() != g.nnz_total * heads:
            raise ValueError("edge must have nnz_total * heads values")
    elif edge is not None:
        raise ValueError("copy_src takes no edge values")
    shape = (g.num_rows,) + tuple(x.shape[1:])
    out = torch.empty(shape, dtype=torch.float32, device=x.device) if out is None else \
        _dev_tensor(out, torch.float32, "out")
    if out.numel() != g.num_rows * F:
        raise ValueError("out has the wrong size")
    if reduce == "max":
        arg = torch.empty(shape, dtype=torch.int32, device=x.device) if arg is None else \
            _dev_tensor(arg, torch.int32, "arg")
        if arg.numel() != g.num_rows * F:
            raise ValueError("arg has the wrong size")
    else:
        arg = None
    st = _lib.fg_gspmm(ctypes.byref(g._c), MSG_OPS[msg], REDUCE_OPS[reduce], heads, dh,
                       _ptr(x), _ptr(edge), _ptr(out), _ptr(arg), _plan_handle(plan), _stream())
    _check(st, "fg_gspmm")
    return (out, arg) if reduce == "max" else out


def gspmm_noalloc(g: Graph, x: torch.Tensor, out: torch.Tensor,
                  arg: Optional[torch.Tensor] = None, edge: Optional[torch.Tensor] = None,
                  msg: str = "copy_src", reduce: str = "sum", heads: int = 1,
                  plan: Optional[Plan] = None):
    """gspmm through fg_gspmm_noalloc: nothing is allocated, neither by the
    library (split-row partials go to its fixed per-device scratch of
    NOALLOC_SCRATCH_BYTES) nor here, so the caller passes ``out`` (and
    ``arg`` for reduce='max').  Same results as gspmm with the same plan.
    Raises FgError (status FG_ERR_SCRATCH_LIMIT) when the plan's partials do
    not fit the scratch.  Calls on one device share the scratch: order them
    on one stream."""
    if msg not in MSG_OPS or reduce not in REDUCE_OPS:
        raise ValueError("unknown msg %r or reduce %r" % (msg, reduce))
    x = _dev_tensor(x, torch.float32, "x")
    if x.shape[0] != g.num_cols:
        raise ValueError("x must have num_cols rows")
    F = int(np.prod(x.shape[1:])) if x.dim() > 1 else 1
    if x.dim() == 3:
        heads = int(x.shape[1])
    if F % heads:
        raise ValueError("feature width not divisible by heads")
    if msg == "src_mul_edge":
        if edge is None:
            raise ValueError("src_mul_edge needs edge values")
        edge = _dev_tensor(edge, torch.float32, "edge")
        if edge.numel() != g.nnz_total * heads:
            raise ValueError("edge must have nnz_total * heads values")
    elif edge is not None:
        raise ValueError("copy_src takes no edge values")
    out = _dev_tensor(out, torch.float32, "out")
    if out.numel() != g.num_rows * F:
        raise ValueError("out has the wrong size")
    if reduce == "max":
        if arg is None:
            raise ValueError("reduce='max' needs arg (nothing is allocated here)")
        arg = _dev_tensor(arg, torch.int32, "arg")
        if arg.numel() != g.num_rows * F:
            raise ValueError("arg has the wrong size")
    elif arg is not None:
        raise ValueError("arg is only written for reduce='max'")
    st = _lib.fg_gspmm_noalloc(ctypes.byref(g._c), MSG_OPS[msg], REDUCE_OPS[reduce], heads,
                               F // heads, _ptr(x), _ptr(edge), _ptr(out), _ptr(arg),
                               _plan_handle(plan), _stream())
    _check(st, "fg_gspmm_noalloc")
    return (out, arg) if reduce == "max" else out


def gsddmm(g: Graph, x_src: torch.Tensor, x_dst: Optional[torch.Tensor] = None, heads: int = 1,
           op: str = "dot", plan: Optional[Plan] = None, out: Optional[torch.Tensor] = None):
    """Generalized SDDMM: out[e, h] = x_src[u, h, :] . x_dst[v, h, :] for every
    stored edge u -> v with id e.  x_dst defaults to x_src (square graphs).
    Returns [nnz_total, H] (or [nnz_total] for H = 1 and 2-D inputs)."""
    if op not in EDGE_OPS:
        raise ValueError("unknown edge op %r" % op)
    x_src = _dev_tensor(x_src, torch.float32, "x_src")
    x_dst = x_src if x_dst is None else _dev_tensor(x_dst, torch.float32, "x_dst")
    if x_src.shape[0] != g.num_cols or x_dst.shape[0] != g.num_rows:
        raise ValueError("x_src needs num_cols rows and x_dst num_rows rows")
    if x_src.shape[1:] != x_dst.shape[1:]:
        raise ValueError("x_src and x_dst must have the same feature shape")
    if x_src.dim() == 3:
        heads = int(x_src.shape[1])
    F = int(np.prod(x_src.shape[1:])) if x_src.dim() > 1 else 1
    if F % heads:
        raise ValueError("feature width not divisible by heads")
    shape = (g.nnz_total, heads) if (heads > 1 or x_src.dim() == 3) else (g.nnz_total,)
    out = torch.empty(shape, dtype=torch.float32, device=x_src.device) if out is None else \
        _dev_tensor(out, torch.float32, "out")
    if out.numel() != g.nnz_total * heads:
        raise ValueError("out has the wrong size")
    st = _lib.fg_gsddmm(ctypes.byref(g._c), EDGE_OPS[op], heads, F // heads, _ptr(x_src),
                        _ptr(x_dst), _ptr(out), _plan_handle(plan), _stream())
    _check(st, "fg_gsddmm")
    return out


def edge_softmax(g: Graph, scores: torch.Tensor, leaky: bool = True, slope: float = 0.2,
                 plan: Optional[Plan] = None, out: Optional[torch.Tensor] = None):
    """Softmax of edge scores [nnz_total] or [nnz_total, H] over each row's
    stored edges, per head, after an optional leaky ReLU."""
    scores = _dev_tensor(scores, torch.float32, "scores")
    if scores.shape[0] != g.nnz_total:
        raise ValueError("scores must have nnz_total rows")
    heads = int(scores.shape[1]) if scores.dim() == 2 else 1
    out = torch.empty_like(scores) if out is None else _dev_tensor(out, torch.float32, "out")
    if out.numel() != scores.numel():
        raise ValueError("out has the wrong size")
    st = _lib.fg_edge_softmax(ctypes.byref(g._c), heads, _ptr(scores), 1 if leaky else 0,
                              float(slope), _ptr(out), _plan_handle(plan), _stream())
    _check(st, "fg_edge_softmax")
    return out


def gsddmm_edge_softmax(g: Graph, x_src: torch.Tensor, x_dst: Optional[torch.Tensor] = None,
                        heads: int = 1, leaky: bool = True, slope: float = 0.2,
                        plan: Optional[Plan] = None, scores: Optional[torch.Tensor] = None,
                        out: Optional[torch.Tensor] = None):
    """gsddmm followed by edge_softmax, fused into one pass where the shape
    allows: returns (scores, attention weights), each [nnz_total] or
    [nnz_total, H]."""
    x_src = _dev_tensor(x_src, torch.float32, "x_src")
    x_dst = x_src if x_dst is None else _dev_tensor(x_dst, torch.float32, "x_dst")
    if x_src.shape[0] != g.num_cols or x_dst.shape[0] != g.num_rows:
        raise ValueError("x_src needs num_cols rows and x_dst num_rows rows")
    if x_src.shape[1:] != x_dst.shape[1:]:
        raise ValueError("x_src and x_dst must have the same feature shape")
    if x_src.dim() == 3:
        heads = int(x_src.shape[1])
    F = int(np.prod(x_src.shape[1:])) if x_src.dim() > 1 else 1
    if F % heads:
        raise ValueError("feature width not divisible by heads")
    shape = (g.nnz_total, heads) if (heads > 1 or x_src.dim() == 3) else (g.nnz_total,)
    res = []
    for name, t in (("scores", scores), ("out", out)):
        t = torch.empty(shape, dtype=torch.float32, device=x_src.device) if t is None else \
            _dev_tensor(t, torch.float32, name)
        if t.numel() != g.nnz_total * heads:
            raise ValueError("%s has the wrong size" % name)
        res.append(t)
    st = _lib.fg_gsddmm_edge_softmax(ctypes.byref(g._c), heads, F // heads, _ptr(x_src),
                                     _ptr(x_dst), 1 if leaky else 0, float(slope), _ptr(res[0]),
                                     _ptr(res[1]), _plan_handle(plan), _stream())
    _check(st, "fg_gsddmm_edge_softmax")
    return res[0], res[1]


def gat_aggregate(g: Graph, x_src: torch.Tensor, x_dst: Optional[torch.Tensor] = None,
                  heads: int = 1, leaky: bool = True, slope: float = 0.2,
                  plan: Optional[Plan] = None, out: Optional[torch.Tensor] = None):
    """Fused gsddmm -> edge_softmax -> gspmm(src_mul_edge, sum): for every row
    v and head h, out[v, h] = sum over in-edges of softmax(leaky(x_src[u, h] .
    x_dst[v, h])) * x_src[u, h], without per-edge intermediates.  Raises
    FgError(FG_ERR_UNSUPPORTED) for shapes the fused kernel does not cover."""
    x_src = _dev_tensor(x_src, torch.float32, "x_src")
    x_dst = x_src if x_dst is None else _dev_tensor(x_dst, torch.float32, "x_dst")
    if x_src.shape[0] != g.num_cols or x_dst.shape[0] != g.num_rows:
        raise ValueError("x_src needs num_cols rows and x_dst num_rows rows")
    if x_src.shape[1:] != x_dst.shape[1:]:
        raise ValueError("x_src and x_dst must have the same feature shape")
    if x_src.dim() == 3:
        heads = int(x_src.shape[1])
    F = int(np.prod(x_src.shape[1:])) if x_src.dim() > 1 else 1
    if F % heads:
        raise ValueError("feature width not divisible by heads")
    shape = (g.num_rows,) + tuple(x_src.shape[1:])
    out = torch.empty(shape, dtype=torch.float32, device=x_src.device) if out is None else \
        _dev_tensor(out, torch.float32, "out")
    if out.numel() != g.num_rows * F:
        raise ValueError("out has the wrong size")
    st = _lib.fg_gat_aggregate(ctypes.byref(g._c), heads, F // heads, _ptr(x_src), _ptr(x_dst),
                               1 if leaky else 0, float(slope), _ptr(out), _plan_handle(plan),
                               _stream())
    _check(st, "fg_gat_aggregate")
    return out


# ----------------------------------------------------------------------------
# backward operators (the backward of gspmm-sum and gsddmm are gsddmm / gspmm
# calls on the graph or its transpose)
# ----------------------------------------------------------------------------


def gspmm_max_backward(g: Graph, arg: torch.Tensor, grad_out: torch.Tensor,
                       x: Optional[torch.Tensor] = None, edge: Optional[torch.Tensor] = None,
                       msg: str = "copy_src", heads: int = 1, plan: Optional[Plan] = None,
                       want_src: bool = True, want_edge: bool = False,
                       grad_src: Optional[torch.Tensor] = None,
                       grad_edge: Optional[torch.Tensor] = None):
    """Gradient of gspmm(..., reduce='max'): grad_out [num_rows, F] (or
    [num_rows, H, dh]) goes to the source of the edge each output element was
    taken from (arg, the forward's edge ids).  Returns grad_src [num_cols, ...]
    and/or grad_edge [nnz_total, H] (src_mul_edge only; needs x).  Graphs with
    explicit edge ids need their plan.  With a plan created with
    ``max_backward=True`` grad_src is summed per source tile in LDS after a
    counting sort instead of with fp32 atomics."""
    if msg not in MSG_OPS:
        raise ValueError("unknown msg %r" % msg)
    grad_out = _dev_tensor(grad_out, torch.float32, "grad_out")
    arg = _dev_tensor(arg, torch.int32, "arg")
    if grad_out.shape[0] != g.num_rows or arg.shape != grad_out.shape:
        raise ValueError("grad_out and arg must be [num_rows, ...] of one shape")
    F = int(np.prod(grad_out.shape[1:])) if grad_out.dim() > 1 else 1
    if grad_out.dim() == 3:
        heads = int(grad_out.shape[1])
    if F % heads:
        raise ValueError("feature width not divisible by heads")
    if msg == "src_mul_edge":
        if edge is None:
            raise ValueError("src_mul_edge needs edge values")
        edge = _dev_tensor(edge, torch.float32, "edge")
        if edge.numel() != g.nnz_total * heads:
            raise ValueError("edge must have nnz_total * heads values")
    elif edge is not None or want_edge:
        raise ValueError("copy_src has no edge values (and no edge gradient)")
    if want_edge:
        if x is None:
            raise ValueError("the edge gradient needs the source features x")
        x = _dev_tensor(x, torch.float32, "x")
        if x.numel() != g.num_cols * F:
            raise ValueError("x must be [num_cols, F]")
    else:
        x = None
    dev = grad_out.device
    if want_src:
        shape = (g.num_cols,) + tuple(grad_out.shape[1:])
        grad_src = torch.empty(shape, dtype=torch.float32, device=dev) if grad_src is None else \
            _dev_tensor(grad_src, torch.float32, "grad_src")
        if grad_src.numel() != g.num_cols * F:
            raise ValueError("grad_src has the wrong size")
    else:
        grad_src = None
    if want_edge:
        grad_edge = torch.empty((g.nnz_total, heads), dtype=torch.float32, device=dev) \
            if grad_edge is None else _dev_tensor(grad_edge, torch.float32, "grad_edge")
        if grad_edge.numel() != g.nnz_total * heads:
            raise ValueError("grad_edge has the wrong size")
    else:
        grad_edge = None
    st = _lib.fg_gspmm_max_backward(ctypes.byref(g._c), MSG_OPS[msg], heads, F // heads,
                                    _ptr(x), _ptr(edge), _ptr(arg), _ptr(grad_out),
                                    _ptr(grad_src), _ptr(grad_edge), _plan_handle(plan),
                                    _stream())
    _check(st, "fg_gspmm_max_backward")
    if want_src and want_edge:
        return grad_src, grad_edge
    return grad_src if want_src else grad_edge


def edge_softmax_backward(g: Graph, out: torch.Tensor, grad_out: torch.Tensor,
                          scores: Optional[torch.Tensor] = None, leaky: bool = True,
                          slope: float = 0.2, plan: Optional[Plan] = None,
                          grad_scores: Optional[torch.Tensor] = None):
    """Gradient of edge_softmax w.r.t. its scores, from its output `out` (the
    attention weights), the upstream gradient and (leaky ReLU only) the
    forward's scores.  grad_scores may be grad_out itself (in place)."""
    out = _dev_tensor(out, torch.float32, "out")
    grad_out = _dev_tensor(grad_out, torch.float32, "grad_out")
    if out.shape[0] != g.nnz_total or grad_out.shape != out.shape:
        raise ValueError("out and grad_out must be [nnz_total(, H)] of one shape")
    heads = int(out.shape[1]) if out.dim() == 2 else 1
    if leaky:
        if scores is None:
            raise ValueError("the leaky ReLU's gradient needs the forward's scores")
        scores = _dev_tensor(scores, torch.float32, "scores")
        if scores.shape != out.shape:
            raise ValueError("scores must have the shape of out")
    else:
        scores = None
    grad_scores = torch.empty_like(out) if grad_scores is None else \
        _dev_tensor(grad_scores, torch.float32, "grad_scores")
    if grad_scores.numel() != out.numel():
        raise ValueError("grad_scores has the wrong size")
    st = _lib.fg_edge_softmax_backward(ctypes.byref(g._c), heads, _ptr(out), _ptr(grad_out),
                                       _ptr(scores), 1 if leaky else 0, float(slope),
                                       _ptr(grad_scores), _plan_handle(plan), _stream())
    _check(st, "fg_edge_softmax_backward")
    return grad_scores


def gsddmm_edge_softmax_backward(g: Graph, x_src: torch.Tensor, x_dst: torch.Tensor,
                                 out: torch.Tensor, scores: Optional[torch.Tensor] = None,
                                 leaky: bool = True, slope: float = 0.2,
                                 plan: Optional[Plan] = None,
                                 grad_scores: Optional[torch.Tensor] = None):
    """The score gradient of an attention layer in one call: the per-head
    gsddmm of x_src [num_cols, H, dh] and x_dst [num_rows, H, dh] (the
    aggregation's upstream gradient), fed into edge_softmax_backward with the
    forward's attention weights `out` [nnz_total, H] (and scores for the
    leaky ReLU).  Returns grad_scores [nnz_total, H]."""
    x_src = _dev_tensor(x_src, torch.float32, "x_src")
    x_dst = _dev_tensor(x_dst, torch.float32, "x_dst")
    out = _dev_tensor(out, torch.float32, "out")
    if x_src.dim() != 3 or x_dst.dim() != 3 or x_src.shape[1:] != x_dst.shape[1:]:
        raise ValueError("x_src and x_dst must be [n, H, dh] with the same H and dh")
    if x_src.shape[0] != g.num_cols or x_dst.shape[0] != g.num_rows:
        raise ValueError("x_src must have num_cols rows and x_dst num_rows rows")
    heads, dh = int(x_src.shape[1]), int(x_src.shape[2])
    if out.numel() != g.nnz_total * heads:
        raise ValueError("out must be [nnz_total, H]")
    if leaky:
        if scores is None:
            raise ValueError("the leaky ReLU's gradient needs the forward's scores")
        scores = _dev_tensor(scores, torch.float32, "scores")
        if scores.numel() != out.numel():
            raise ValueError("scores must have the size of out")
    else:
        scores = None
    grad_scores = torch.empty((g.nnz_total, heads), dtype=torch.float32, device=out.device) \
        if grad_scores is None else _dev_tensor(grad_scores, torch.float32, "grad_scores")
    if grad_scores.numel() != out.numel():
        raise ValueError("grad_scores has the wrong size")
    st = _lib.fg_gsddmm_edge_softmax_backward(ctypes.byref(g._c), heads, dh, _ptr(x_src),
                                              _ptr(x_dst), _ptr(out), _ptr(scores),
                                              1 if leaky else 0, float(slope),
                                              _ptr(grad_scores), _plan_handle(plan), _stream())
    _check(st, "fg_gsddmm_edge_softmax_backward")
    return grad_scores


# ----------------------------------------------------------------------------
# MLP aggregation
# ----------------------------------------------------------------------------


def dense_matmul(x: torch.Tensor, w: torch.Tensor, out: Optional[torch.Tensor] = None):
    """y = x w on the matrix cores: x [n, d_in], w [d_in, d_out] fp32."""
    x = _dev_tensor(x, torch.float32, "x")
    w = _dev_tensor(w, torch.float32, "w")
    if x.dim() != 2 or w.dim() != 2 or x.shape[1] != w.shape[0]:
        raise ValueError("x must be [n, d_in] and w [d_in, d_out]")
    n, d_in = x.shape
    d_out = w.shape[1]
    out = torch.empty((n, d_out), dtype=torch.float32, device=x.device) if out is None else \
        _dev_tensor(out, torch.float32, "out")
    if out.numel() != n * d_out:
        raise ValueError("out has the wrong size")
    _check(_lib.fg_dense_matmul(n, d_in, d_out, _ptr(x), _ptr(w), _ptr(out), _stream()),
           "fg_dense_matmul")
    return out


def mlp_aggregate(g: Graph, x_src: torch.Tensor, weight: torch.Tensor,
                  x_dst: Optional[torch.Tensor] = None, plan: Optional[Plan] = None,
                  out: Optional[torch.Tensor] = None, arg: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None):
    """MLP aggregation: out[v, i] = max over in-edges of relu(((x_src[u] +
    x_dst[v]) weight)[i]) and the edge id of each maximum.  x_dst defaults to
    x_src (square graphs).  workspace: (num_cols + num_rows) * d_out floats
    of scratch, allocated here when not given."""
    x_src = _dev_tensor(x_src, torch.float32, "x_src")
    x_dst = x_src if x_dst is None else _dev_tensor(x_dst, torch.float32, "x_dst")
    weight = _dev_tensor(weight, torch.float32, "weight")
    if weight.dim() != 2:
        raise ValueError("weight must be [d_in, d_out]")
    d_in, d_out = weight.shape
    if x_src.shape != (g.num_cols, d_in) or x_dst.shape != (g.num_rows, d_in):
        raise ValueError("x_src must be [num_cols, d_in] and x_dst [num_rows, d_in]")
    dev = x_src.device
    out = torch.empty((g.num_rows, d_out), dtype=torch.float32, device=dev) if out is None else \
        _dev_tensor(out, torch.float32, "out")
    arg = torch.empty((g.num_rows, d_out), dtype=torch.int32, device=dev) if arg is None else \
        _dev_tensor(arg, torch.int32, "arg")
    if out.numel() != g.num_rows * d_out or arg.numel() != g.num_rows * d_out:
        raise ValueError("out / arg have the wrong size")
    nws = (g.num_cols + g.num_rows) * d_out
    workspace = torch.empty(max(nws, 1), dtype=torch.float32, device=dev) if workspace is None \
        else _dev_tensor(workspace, torch.float32, "workspace")
    if workspace.numel() < nws:
        raise ValueError("workspace needs (num_cols + num_rows) * d_out floats")
    st = _lib.fg_mlp_aggregate(ctypes.byref(g._c), d_in, d_out, _ptr(x_src), _ptr(x_dst),
                               _ptr(weight), _ptr(out), _ptr(arg), _ptr(workspace),
                               _plan_handle(plan), _stream())
    _check(st, "fg_mlp_aggregate")
    return out, arg


__all__ = ["Graph", "Plan", "gspmm", "gsddmm", "edge_softmax", "gsddmm_edge_softmax",
           "gat_aggregate",
           "gspmm_max_backward", "edge_softmax_backward", "dense_matmul", "mlp_aggregate",
           "schedule_host", "FgError", "status_string", "LIB_PATH"]
