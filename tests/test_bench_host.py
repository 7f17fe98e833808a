"""Host-side pieces of bench.py (no GPU): the single-GPU guard, the
algorithmic byte models against the figures the design notes quote, the
oracle row sampler and the CPU-baseline record."""
import importlib.util
import os
import subprocess
import sys

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_byte_models_power_law_d128(bench):
    """N = 232,965, E = 114.6M, d = 128: 59.71 GB for the weighted gSpMM and
    SDDMM, 59.37 GB for the max (value + arg), 0.92 GB for edge softmax."""
    n, e, d = 232_965, 114_600_000, 128
    assert round(bench.bytes_spmm(n, e, d, 1, weighted=True) / 1e9, 2) == 59.71
    assert round(bench.bytes_spmm(n, e, d, 1, argmax=True) / 1e9, 2) == 59.37
    assert round(bench.bytes_sddmm(n, e, d, 1) / 1e9, 2) == 59.71
    assert round(bench.bytes_softmax(n, e, 1) / 1e9, 2) == 0.92
    # per-edge gather term dominates: 4 E d
    assert bench.bytes_spmm(n, e, d, 1) - bench.bytes_spmm(n, e, d - 1, 1) == 4 * e + 4 * n


def test_byte_models_attention_and_training(bench):
    """Clustered graph (N = 132,534, E = 39.76M, 8 heads of 16): 21.86 GB for
    per-head SDDMM and for the score-weighted gSpMM, 2.55 GB for the 8-head
    softmax (scores read once, weights written once); training graph
    (2^20 vertices, 2^25 edges, d = 256): 35.57 GB for gSpMM, 35.71 GB for
    SDDMM."""
    n, e = 132_534, 39_760_200
    assert round(bench.bytes_sddmm(n, e, 128, 8) / 1e9, 2) == 21.86
    assert round(bench.bytes_spmm(n, e, 128, 8, weighted=True) / 1e9, 2) == 21.86
    assert round(bench.bytes_softmax(n, e, 8) / 1e9, 2) == 2.55
    assert round(bench.bytes_spmm(1 << 20, 1 << 25, 256, 1) / 1e9, 2) == 35.57
    assert round(bench.bytes_sddmm(1 << 20, 1 << 25, 256, 1) / 1e9, 2) == 35.71


def test_row_sample_reaches_its_edge_target(bench):
    c = synth.make_config("rmat_233k_115m", scale_down=256).csr
    rows, ne = bench._row_sample(c, 20_000, 5)
    assert np.all(np.diff(rows) > 0) and rows.size <= c.num_rows
    assert ne == int(c.degrees()[rows].sum())
    # the smallest random prefix of rows holding at least the target
    assert ne >= 20_000 and ne - int(c.degrees()[rows].max()) < 20_000
    assert np.array_equal(bench._row_sample(c, 20_000, 5)[0], rows)  # seeded


def test_cpu_baseline_record(bench):
    """The record's rate is total FLOP over total time of the timed passes."""
    calls = []

    def fake_sample(edges_target):
        calls.append(edges_target)
        return 0.05, int(1e8), "%d rows" % edges_target

    rec = bench._cpu_baseline(fake_sample, 0.2, 3)
    assert rec["unit"] == "GFLOP/s" and rec["cores"] == 3 and rec["kind"] == "oracle"
    assert rec["value"] == pytest.approx(1e8 / 0.05 / 1e9)
    assert calls[0] == 200_000 and calls[1] == 2_000_000 and len(calls) >= 6
    assert "passes" in rec["sample"] and rec["host"]["logical_cpus"] == os.cpu_count()


def test_simple_graph_keeps_one_edge_per_pair(bench):
    """--simple-graph: every (destination, source) pair once, first copies
    kept, rows and their order otherwise unchanged."""
    rng = np.random.default_rng(3)
    dst = rng.integers(0, 50, 3000)
    src = rng.integers(0, 20, 3000)
    csr = synth.coo_to_csr(dst, src, 60, 20)
    simple, keep = bench.simple_graph(csr)
    synth.check_csr(simple)
    rows = synth.csr_rows(csr)
    pairs = set(zip(rows.tolist(), csr.indices.tolist()))
    srows = synth.csr_rows(simple)
    spairs = list(zip(srows.tolist(), simple.indices.tolist()))
    assert len(spairs) == len(set(spairs)) == len(pairs) and set(spairs) == pairs
    # the kept positions are the first copy of each pair, in storage order
    first = {}
    for q, pr in enumerate(zip(rows.tolist(), csr.indices.tolist())):
        first.setdefault(pr, q)
    assert np.array_equal(np.nonzero(keep)[0], np.array(sorted(first.values())))
    assert simple.num_rows == csr.num_rows and simple.num_cols == csr.num_cols


def test_roofline_extras_from_counters(bench):
    """Counter-grounded roofline figures: traffic rate and fraction of 8 TB/s,
    and the vector-memory ceiling from read instructions, the gather floor in
    cycles and the kernel's cycles per CU."""
    per_op = {"k": {"ms_mean": 2.0}}
    # 51.2M instructions / 256 CUs * 16 cycles = 3.2M of the kernel's 4M cycles
    ctr = {"hbm_bytes_per_launch": 12_000_000_000, "read_instructions": 51_200_000,
           "gui_active_cycles": 32_000_000, "ta_busy_cycles": 921_600_000}
    ex = bench.roofline_extras(per_op, "k", ctr, 16.0)
    assert ex["traffic_gbs"] == 6000.0 and ex["traffic_frac"] == 0.75
    v = ex["vmem"]
    assert v["kernel_cycles_per_cu"] == 4_000_000 and v["frac"] == 0.8
    assert v["ceiling_ms"] == 1.6 and v["ta_busy"] == 0.9
    assert bench.roofline_extras(per_op, "k", None, 16.0) == {}
    assert "vmem" not in bench.roofline_extras(per_op, "k", ctr, None)
