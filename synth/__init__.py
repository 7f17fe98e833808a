"""Seeded synthetic graphs and feature tensors.

This package is shared by the CPU oracle's tests and by the GPU path's tests
and benchmark.  It only draws random structure and values and lays them out
(COO -> CSR sorted by destination, CSR -> CSC); it holds none of the
aggregation, dot-product or softmax arithmetic of the method.
"""
from .graphs import (  # noqa: F401
    CSR,
    Workload,
    coo_to_csr,
    csr_to_csc,
    csr_rows,
    sha256,
    check_csr,
    uniform_graph,
    fixed_indegree_graph,
    rmat_graph,
    clustered_graph,
    two_class_graph,
    make_config,
    small_random_graph,
    CONFIG_NAMES,
)
