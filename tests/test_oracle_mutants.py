"""Planted mistakes in a copy of the oracle must each be caught by at least one pin.

Each mutant is the oracle's C source with one plausible mistake (a dropped
term, a wrong index, a wrong sign, a wrong divisor, a clipped max, a lost
weight, a wrong empty value). It is compiled with gcc into a temporary library
and the pins of ``oracle_pins.py`` run against it in a child process, so a
mutant that crashes counts as caught too. Nothing here touches the GPU.
"""
import os
import subprocess
import sys
import tempfile

import pytest

import oracle

MUTANTS = {
    "drop_last_term": ("for (int64_t i = b; i < e; ++i) acc += (double)term",
                       "for (int64_t i = b; i < e - 1; ++i) acc += (double)term"),
    "boundary_off_by_one": ("while (i < nnz && idx[i] < s) ++i;",
                            "while (i < nnz && idx[i] <= s) ++i;"),
    "max_clipped_at_zero": ("float m = term(rows, F, col, w, b, f);",
                            "float m = 0.0f;"),
    "mean_wrong_divisor": ("if (op == OR_MEAN) acc = acc / (double)count;",
                           "if (op == OR_MEAN) acc = acc / (double)(count + 1);"),
    "weight_ignored": ("float t = w[e] * x; /* one fp32 multiply */",
                       "float t = x;"),
    "gather_ignores_col": ("float x = rows[col[e] * F + f];",
                           "float x = rows[(e % n_rows_guard) * F + f];"),
    "sign_flip": ("for (int64_t i = b; i < e; ++i) acc += (double)term",
                  "for (int64_t i = b; i < e; ++i) acc -= (double)term"),
    "empty_value_wrong": ("result = 0.0f; /* empty segment */",
                          "result = -1.0f; /* empty segment */"),
    "columns_reversed": ("out[s * F + f] = result;",
                         "out[s * F + (F - 1 - f)] = result;"),
    "max_keeps_first": ("m = maximum(m, t);", "if (i < b) m = maximum(m, t);"),
    "max_drops_nan": ("    if (isnan(a)) return a;\n", ""),
    "max_zero_sign_by_order": ("if (a == b) return signbit(a) ? b : a;", "if (a == b) return a;"),
    "stats_var_unsquared": ("v += d * d;", "v += d;"),
    "bwd_mean_no_divide": ("r = (float)(g / (double)(e - b));", "r = (float)g;"),
    "bwd_max_last_member": ("} else if (!found && src[i * F + f] == out[s * F + f]) {",
                            "} else if (src[i * F + f] == out[s * F + f]) {"),
    "bwd_grad_w_wrong_factor": ("double tx = coef * g, tw = g * x;", "double tx = coef * g, tw = coef * x;"),
    "bwd_grad_x_by_row": ("if (grad_X) grad_X[col[e] * F + f] += tx;",
                          "if (grad_X) grad_X[(r % n_x) * F + f] += tx;"),
    "bwd_abs_x_signed": ("tx = fabs(tx);", "tx = +tx;"),
    "bwd_abs_w_signed": ("tw = fabs(tw);", "tw = +tw;"),
}

RUNNER = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle
from oracle_pins import ALL_PINS
impl = oracle.OracleLib({lib!r})
failed = []
for pin in ALL_PINS:
    try:
        pin(impl)
    except Exception as e:  # AssertionError or an oracle error both count
        failed.append(pin.__name__)
print("FAILED:" + ",".join(failed))
"""


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(oracle.SOURCE).read()
    assert src.count(old) >= 1, f"mutation anchor missing for {name}"
    mutated = src.replace(old, new, 1)
    if "n_rows_guard" in new:
        # a safe stand-in index for the ignored column (rows of X, never out of bounds)
        mutated = mutated.replace("static float term(const float *rows, int64_t F,",
                                  "static int64_t n_rows_guard = 1;\nstatic float term(const float *rows, int64_t F,")
        mutated = mutated.replace("segment_starts(row, nnz, R, start);",
                                  "segment_starts(row, nnz, R, start); n_rows_guard = n_x > 0 ? n_x : 1;")
    csrc = tmp_path / "mutant.c"
    csrc.write_text(mutated)
    lib = str(tmp_path / "libmutant.so")
    oracle.build(str(csrc), lib)
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = RUNNER.format(root=root, tests=os.path.join(root, "tests"), lib=lib)
    proc = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    if proc.returncode != 0:
        return  # the mutant crashed the pins: caught
    line = [l for l in proc.stdout.splitlines() if l.startswith("FAILED:")][-1]
    failed = [f for f in line[len("FAILED:"):].split(",") if f]
    assert failed, f"mutant {name} passed every pin"
