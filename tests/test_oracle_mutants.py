"""The oracle's pins are strong enough to catch plausible mistakes.

Each mutant is a copy of oracle/fgref.c with one planted mistake (a dropped
term, a wrong index or sign, a swapped operand, a wrong tie-break).  The pin
suite (tests/test_oracle_pins.py) runs against every mutant in its own
process, with FGREF_LIB pointing the oracle shim at the mutant's library; the
suite must fail for each one.  CPU only; nothing here touches the GPU path.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "fgref.c")

# (name, original text, planted mistake[, "all" to replace every occurrence])
MUTANTS = [
    ("spmm_source_is_position", "const int64_t u = indices[p];\n          const int64_t e = edge_ids ? edge_ids[p] : p;\n          if (u < 0",
     "const int64_t u = p % num_cols;\n          const int64_t e = edge_ids ? edge_ids[p] : p;\n          if (u < 0"),
    ("spmm_weight_dropped", "m = edge_val[e * H + h] * m;", "m = m;"),
    ("spmm_weight_head_ignored", "m = edge_val[e * H + h] * m;", "m = edge_val[e * H] * m;"),
    ("spmm_weight_by_position", "m = edge_val[e * H + h] * m;", "m = edge_val[p * H + h] * m;"),
    ("spmm_sum_sign", "acc += (double)m;", "acc -= (double)m;"),
    ("spmm_last_edge_dropped", "for (int64_t p = p0; p < p1; ++p) {\n          const int64_t u = indices[p];",
     "for (int64_t p = p0; p < p1 - 1; ++p) {\n          const int64_t u = indices[p];"),
    ("max_tie_to_largest_id", "(m == best && e < best_e)", "(m == best && e > best_e)"),
    ("max_arg_is_position", "best_e = (int32_t)e;", "best_e = (int32_t)p;"),
    ("sddmm_operands_from_source", "(double)xd[v * F + h * dh + k]", "(double)xd[u * F + h * dh + k]"),
    ("sddmm_head_offset_dropped", "(double)xs[u * F + h * dh + k]", "(double)xs[u * F + k]"),
    ("sddmm_written_by_position", "out[e * H + h] = (float)acc;\n        if (term_norm) term_norm[e * H + h]",
     "out[p * H + h] = (float)acc;\n        if (term_norm) term_norm[e * H + h]"),
    ("softmax_leaky_skipped_in_sum", "        z += exp(s - m);", "        z += exp(scores[e * H + h] - m);"),
    # flipped in every pass (flipping it in the max pass alone only moves the
    # stabilising shift, which leaves the result unchanged: not a mistake)
    ("softmax_leaky_condition_flipped", "if (apply_leaky_relu && !(s > 0.0))",
     "if (apply_leaky_relu && (s > 0.0))", "all"),
    ("max_bwd_to_destination", "const int64_t u = indices[pos[e]];", "const int64_t u = v % num_cols;"),
    ("max_bwd_source_by_id_not_position", "const int64_t u = indices[pos[e]];", "const int64_t u = indices[e];"),
    ("max_bwd_weight_dropped", "? (double)edge_val[e * H + h] * g : g;", "? g : g;"),
    ("max_bwd_edge_grad_without_x", "const double te = (double)x[u * F + f] * g;", "const double te = g;"),
    ("max_bwd_grad_by_selection_index", "const double g = grad_out[v * F + f];", "const double g = grad_out[i * F + f];"),
    ("softmax_bwd_not_centred", "grad_scores[e * H + h] = (float)(a * (g - c) * lf);",
     "grad_scores[e * H + h] = (float)(a * g * lf);"),
    ("softmax_bwd_leaky_factor_dropped", "grad_scores[e * H + h] = (float)(a * (g - c) * lf);",
     "grad_scores[e * H + h] = (float)(a * (g - c));"),
    ("softmax_bwd_centre_unweighted", "c += a * (double)grad_out[e * H + h];",
     "c += (double)grad_out[e * H + h];"),
    ("mlp_dst_feature_dropped", "const double h = (double)xs[u * d_in + k] + (double)xd[v * d_in + k];",
     "const double h = (double)xs[u * d_in + k];"),
    ("mlp_weight_transposed", "w[k * d_out + i]", "w[i * d_in + k]", "all"),
    ("mlp_relu_dropped", "const double m = t > 0.0 ? t : 0.0;", "const double m = t;"),
    ("mlp_tie_to_largest_id", "(m == best && e < best_e)) {\n          best = m;\n          best_e = (int32_t)e;\n          best_scale",
     "(m == best && e > best_e)) {\n          best = m;\n          best_e = (int32_t)e;\n          best_scale"),
    ("dense_matmul_weight_transposed", "(double)w[k * d_out + j]", "(double)w[j * d_in + k]"),
    ("dense_matmul_last_term_dropped", "for (int64_t k = 0; k < d_in; ++k) acc +=",
     "for (int64_t k = 0; k < d_in - 1; ++k) acc +="),
    ("max_nan_not_minus_inf", "if (red == RED_MAX && isnan(m)) m = -INFINITY;", ""),
    ("softmax_off_normaliser", "out[e * H + h] = (float)(exp(s - m) / z);", "out[e * H + h] = (float)(exp(s - m) / (z + 1e-3));"),
]


def _run_mutant(tmpdir, name, old, new, where="first"):
    src = open(SRC).read()
    assert src.count(old) >= 1, name
    mut_src = os.path.join(tmpdir, name + ".c")
    with open(mut_src, "w") as f:
        f.write(src.replace(old, new) if where == "all" else src.replace(old, new, 1))
    lib = os.path.join(tmpdir, name + ".so")
    sys.path.insert(0, ROOT)
    from oracle.fgref import compile_oracle

    compile_oracle(mut_src, lib)
    env = dict(os.environ, FGREF_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, r.returncode


def test_every_mutant_is_caught(tmp_path):
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda m: _run_mutant(str(tmp_path), *m), MUTANTS))
    survivors = [name for name, rc in results if rc == 0]
    assert not survivors, "pins did not catch: %s" % survivors


def test_unmutated_oracle_passes_the_same_way(tmp_path):
    """Control: the copy-compile-subprocess route itself passes on the real source."""
    name, rc = _run_mutant(str(tmp_path), "control", "/*", "/*")
    assert rc == 0
