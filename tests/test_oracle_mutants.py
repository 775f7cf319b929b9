"""Planted mistakes in the oracle must fail its pins (no GPU).

Each mutant is a copy of oracle/softmax_f64.c with one plausible mistake
(a dropped term, a wrong sign, a wrong index or stride, a wrong operation),
built with the same gcc line into a temporary directory.  Every mutation keeps
all memory accesses in bounds.  The transposed-operand mistake is planted in
the Python wrapper's orientation instead.
"""
import os

import pytest

import oracle
from oracle_pins import run_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "softmax_f64.c")

MUTANTS = {
    "no_max_subtraction": ("double e = exp(x[j] - m);", "double e = exp(x[j]);"),
    "wrong_sign": ("double e = exp(x[j] - m);", "double e = exp(m - x[j]);"),
    "multiply_not_divide": ("y[j] = y[j] / s;", "y[j] = y[j] * s;"),
    "min_not_max": ("if (x[j] > m)", "if (x[j] < m)"),
    "sum_starts_at_one": ("double s = 0.0;", "double s = 1.0;"),
    "sum_keeps_last_term": ("s += e;", "s = e;"),
    "first_term_dropped": ("for (int64_t j = 0; j < cols; ++j) {\n        double e",
                           "for (int64_t j = 1; j < cols; ++j) {\n        double e"),
    "reversed_output_index": ("y[j] = e;", "y[cols - 1 - j] = e;"),
    "wrong_input_row_stride": (
        "oracle_row(job->x + r * job->cols, job->y + r * job->cols, job->cols);",
        "oracle_row(job->x + r, job->y + r * job->cols, job->cols);"),
    "thread_rows_lost": ("jobs[t].row_end = rows * (t + 1) / threads;",
                         "jobs[t].row_end = rows * (t + 1) / threads - (t < threads - 1);"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_fails_a_pin(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = oracle.load(oracle.build(str(path), str(tmp_path / f"lib{name}.so")))
    fails = run_pins(lambda x, threads=1: oracle.softmax_f64(x, threads=threads, lib=lib))
    assert fails, f"mutant {name} passed every pin"


def test_transposed_orientation_fails_a_pin():
    def along_columns(x, threads=1):
        import numpy as np
        x = np.asarray(x, dtype=np.float64)
        return oracle.softmax_f64(np.ascontiguousarray(x.T), threads=threads).T
    assert run_pins(along_columns)
