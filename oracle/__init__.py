"""CPU oracle (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path never does: it fails when its own HIP
library is missing instead of falling back here.
"""
from .fgref import (  # noqa: F401
    build,
    lib_path,
    gspmm,
    gsddmm,
    edge_softmax,
    gspmm_max_backward,
    edge_softmax_backward,
    mlp_aggregate,
    dense_matmul,
    max_threads,
    set_num_threads,
    MSG_COPY_SRC,
    MSG_SRC_MUL_EDGE,
    RED_SUM,
    RED_MAX,
)
