"""Plant plausible mistakes in a copy of the oracle source (on the CPU) and
check that the pin suite catches every one. Each mutant runs in its own
subprocess, so one that crashes is also reported as caught."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, original text, mutated text): each original must occur exactly once.
MUTATIONS = [
    ("drop_c_term", " + c * A2[i * n + j];", ";"),
    ("flip_b_sign", "+ b * A[i * n + j]", "- b * A[i * n + j]"),
    ("a_times_A_not_I", "(i == j ? a : 0.0)", "a * A[i * n + j]"),
    ("square_dropped", "matmul(A, A, A2, n, n, n);", "memcpy(A2, A, sizeof(double) * n * n);"),
    ("right_multiply", "matmul(M, X, Xn, n, n, m);", "matmul(X, M, Xn, n, n, m);"),
    ("gram_wrong_index", "X[i * m + k] * X[j * m + k]", "X[i * m + k] * X[k * m + j]"),
    ("norm_squared", "X[i] = X[i] / nrm;", "X[i] = X[i] / nrm2;"),
    ("one_step_short", "for (int k = 0; k < K; ++k) {", "for (int k = 1; k < K; ++k) {"),
    ("no_transpose_back", "Y[i * ld_out + j] = transpose ? X[j * m + i] : X[i * m + j];",
     "Y[i * ld_out + j] = X[i * W + j];"),
    ("pad_with_ones", "? A[gi * ld_in + gj] : 0.0;", "? A[gi * ld_in + gj] : 1.0;"),
    ("tile_index_colmajor", "int64_t r = tile_id / C, cc = tile_id % C;",
     "int64_t r = tile_id % R, cc = tile_id / R;"),
    ("floor_tile_count", "    int64_t R = (H + Th - 1) / Th, C = (W + Tw - 1) / Tw;\n    int status",
     "    int64_t R = H / Th, C = W / Tw;\n    int status"),
    ("rect_tile_rows_cols_swapped", "int64_t gi = r * Th + i, gj = cc * Tw + j;\n            S[",
     "int64_t gi = r * Tw + i, gj = cc * Th + j;\n            S["),
    ("zero_tile_not_zero", "if (nrm == 0.0) {", "if (nrm < 0.0) {"),
    ("step_momentum_no_beta", "Mt[i] = beta * Mt[i] + G[i];", "Mt[i] = Mt[i] + G[i];"),
    ("step_nesterov_old_buffer",
     "Mt[i] = beta * Mt[i] + G[i];\n        Ghat[i] = nesterov ? G[i] + beta * Mt[i] : Mt[i];",
     "Ghat[i] = nesterov ? G[i] + beta * Mt[i] : beta * Mt[i] + G[i];\n        Mt[i] = beta * Mt[i] + G[i];"),
    ("step_nesterov_flag_flipped", "nesterov ? G[i] + beta * Mt[i] : Mt[i]", "nesterov ? Mt[i] : G[i] + beta * Mt[i]"),
    ("step_tau_no_sqrt", "sqrt((double)(full ? big : T))", "(double)(full ? big : T)"),
    ("step_branch_on_min", "int64_t big = H > W ? H : W;", "int64_t big = H < W ? H : W;"),
    ("step_decay_sign", "(1.0 - lr * lambda) * Wt[i]", "(1.0 + lr * lambda) * Wt[i]"),
    ("step_update_sign", "Wt[i] - lr * tau * U[i]", "Wt[i] + lr * tau * U[i]"),
]


def _run_pins(lib_path):
    env = dict(os.environ, PYTHONPATH=os.pathsep.join([ROOT, os.path.join(ROOT, "tests")]))
    return subprocess.run([sys.executable, os.path.join(ROOT, "tests", "oracle_pins.py"), lib_path],
                          env=env, capture_output=True, text=True, timeout=300)


def test_unmutated_copy_passes(tmp_path):
    lib = oracle.build(output=str(tmp_path / "liboracle_copy.so"))
    res = _run_pins(lib)
    assert res.returncode == 0, res.stdout + res.stderr


@pytest.mark.parametrize("name,orig,mut", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutant_is_caught(tmp_path, name, orig, mut):
    src = open(oracle.SOURCE).read()
    assert src.count(orig) == 1, f"mutation site for {name} not found exactly once"
    mutated = tmp_path / f"mutant_{name}.c"
    mutated.write_text(src.replace(orig, mut))
    lib = oracle.build(source=str(mutated), output=str(tmp_path / f"libmutant_{name}.so"))
    res = _run_pins(lib)
    assert res.returncode != 0, f"mutant {name} passed every pin:\n{res.stdout}"
