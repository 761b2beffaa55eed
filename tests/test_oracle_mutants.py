"""Plants plausible mistakes in a copy of the oracle (on the CPU) and checks that the
pins reject every one of them.  The real oracle source is never modified."""
import os
import shutil
import subprocess
import tempfile

import pytest

import _pins
import oracle

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

# (name, text in oracle.c, replacement): each is a mistake a careful reader might make
MUTANTS = [
    ("drop_last_term", "p < row_ptr[i + 1]; ++p) {\n      const double w",
     "p < row_ptr[i + 1] - 1; ++p) {\n      const double w"),
    ("wrong_sign", "acc[n] += t;", "acc[n] -= t;"),
    ("wrong_B_row", "const float* brow = B + (size_t)col_idx[p] * N;\n      for (int32_t n = 0; n < N; ++n) {\n        const double t",
     "const float* brow = B + (size_t)col_idx[row_ptr[i]] * N;\n      for (int32_t n = 0; n < N; ++n) {\n        const double t"),
    ("bias_dropped", "acc[n] = act_f64(acc[n] + bi, epi);", "acc[n] = act_f64(acc[n], epi);"),
    ("bias_wrong_row", "const double bi = bias ? (double)bias[i] : 0.0;",
     "const double bi = bias ? (double)bias[0] : 0.0;"),
    ("gelu_tanh_approx", "return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));",
     "return 0.5 * x * (1.0 + tanh(0.7978845608028654 * (x + 0.044715 * x * x * x)));"),
    ("gelu_no_sqrt2", "return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));",
     "return 0.5 * x * (1.0 + erf(x));"),
    ("relu_identity", "if (epi == 1) return x > 0.0 ? x : 0.0;", "if (epi == 1) return x;"),
    ("bound_signed", "bnd[n] += fabs(t);", "bnd[n] += t;"),
    ("reorder_first_sparsest", "if (nx > nf) first = x;", "if (nx < nf) first = x;"),
    ("reorder_against_first_row", "const int32_t prev = perm_out[i - 1];",
     "const int32_t prev = perm_out[0];"),
    ("reorder_index_only_ties", "(ov == best_ov && xn > best_nnz)", "(0)"),
    ("reorder_last_index_ties", "(ov == best_ov && xn > best_nnz)", "(ov == best_ov && xn >= best_nnz)"),
    ("reorder_merge_wrong_advance", "} else if (a[i] < b[j]) {", "} else if (a[i] > b[j]) {"),
    ("reorder_fewest_overlap", "if (ov > best_ov ||", "if (best_ov < 0 || ov < best_ov ||"),
    ("conv_flipped_rows", "int32_t yy = y + ky - 1, xx = x + kx - 1;",
     "int32_t yy = y - ky + 1, xx = x + kx - 1;"),
    ("conv_swapped_taps", "const int32_t i = tap / 9, ky = (tap % 9) / 3, kx = tap % 3;",
     "const int32_t i = tap / 9, ky = tap % 3, kx = (tap % 9) / 3;"),
    ("conv_clamped_border", "if (yy < 0 || yy >= H || xx < 0 || xx >= W) continue;",
     "if (yy < 0 || yy >= H || xx < 0 || xx >= W) { yy = yy < 0 ? 0 : (yy >= H ? H - 1 : yy); xx = xx < 0 ? 0 : (xx >= W ? W - 1 : xx); }"),
    ("conv_bias_dropped", "C_out[at] = act_f64(acc + bo, epi);", "C_out[at] = act_f64(acc, epi);"),
    ("conv_first_image", "X[i * plane + ((size_t)yy * W + xx) * NB + b]", "X[i * plane + ((size_t)yy * W + xx) * NB]"),
    # mistakes each of which a named pin must reject on its own
    ("bias_halved", "const double bi = bias ? (double)bias[i] : 0.0;",
     "const double bi = bias ? 0.5 * (double)bias[i] : 0.0;", "check_bias_linearity"),
    ("bias_squared", "const double bi = bias ? (double)bias[i] : 0.0;",
     "const double bi = bias ? (double)bias[i] * fabs((double)bias[i]) : 0.0;", "check_bias_linearity"),
    ("gelu_even_erf", "return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));",
     "return 0.5 * x * (1.0 + erf(fabs(x) / sqrt(2.0)));", "check_gelu_odd_part"),
    ("gelu_cdf_not_one", "return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));",
     "return 0.5 * x * (1.000001 + erf(x / sqrt(2.0)));", "check_gelu_odd_part"),
]


@pytest.fixture(scope="module")
def workdir():
    d = tempfile.mkdtemp(prefix="oracle_mut_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_mutant(workdir, mutant):
    name, old, new = mutant[:3]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    path = os.path.join(workdir, f"{name}.c")
    open(path, "w").write(src.replace(old, new))
    so = os.path.join(workdir, f"lib{name}.so")
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-o", so, path, "-lm"],
                   check=True)
    lib = oracle.load(so)
    fails = _pins.run_all(lib)
    assert fails, f"no pin rejects the planted mistake {name}"
    if len(mutant) > 3:  # this pin alone must see the mistake
        assert getattr(_pins, mutant[3])(lib), f"{mutant[3]} does not reject {name}"
