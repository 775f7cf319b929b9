"""The fp64 oracle against its pins (no GPU).

The oracle (oracle/softmax_f64.c) is plain C; everything here checks it
against facts it does not compute itself: a 50-digit brute force with a
different formula, hand-derived closed forms, invariants, independent library
implementations, and closed forms that hold at the real workload shapes.
"""
import numpy as np
import pytest

import oracle
from oracle_pins import brute_force_rows, run_pins
from paper_2607_23089_amd import workloads as W


def test_oracle_builds_and_loads():
    path = oracle.build()
    lib = oracle.load(path)
    assert hasattr(lib, "oracle_softmax_f64")


def test_oracle_passes_every_pin():
    fails = run_pins(lambda x, threads=1: oracle.softmax_f64(x, threads=threads))
    assert fails == []


def test_brute_force_reference_itself():
    # The brute force must agree with a case computed by hand:
    # softmax([0, ln 4]) = [1/5, 4/5].
    v = brute_force_rows(np.array([[0.0, np.log(4.0)]]))
    assert abs(v[0, 0] - 0.2) < 1e-16 and abs(v[0, 1] - 0.8) < 2e-16


@pytest.mark.parametrize("shape", [(0, 5), (3, 0), (0, 0)])
def test_empty(shape):
    y = oracle.softmax_f64(np.zeros(shape))
    assert y.shape == shape


def test_one_dimensional_input_is_one_row():
    y = oracle.softmax_f64(np.array([0.0, 0.0, 0.0, 0.0]))
    assert y.shape == (1, 4) and np.all(y == 0.25)


def test_widening_is_exact():
    bits = np.array([0x3f80, 0xc0a0, 0x7f80, 0xff80, 0x0001, 0x461c], dtype=np.uint16)
    v = oracle.widen_bf16_bits(bits)
    assert v[0] == 1.0 and v[1] == -5.0
    assert v[2] == np.inf and v[3] == -np.inf
    assert v[4] == np.ldexp(1.0, -133)          # smallest bf16 subnormal
    assert v[5] == 9984.0                       # 1e4 rounded to bf16
    f = np.array([1.5, -np.inf, 3.0e-45], dtype=np.float32)
    assert np.array_equal(oracle.widen_f32(f), f.astype(np.float64))


def test_closed_form_vocab_rows():
    # Rows of the vocab workload's shape: every non-outlier entry sits more
    # than 745 below the row maximum 9984, so exp underflows to exactly 0 in
    # fp64 and the oracle must give exactly 1/k at the k entries equal to the
    # maximum and 0 elsewhere.
    w = W.WORKLOADS["vocab_4096x151936"]
    x = W.make_input(w, rows=3)
    v = oracle.widen_bf16_bits(W.to_bits_numpy(x))
    y = oracle.softmax_f64(v, threads=3)
    for r in range(v.shape[0]):
        mx = v[r].max()
        assert mx == 9984.0
        k = int(np.count_nonzero(v[r] == mx))
        assert np.all(y[r][v[r] == mx] == 1.0 / k)
        assert np.all(y[r][v[r] != mx] == 0.0)


def test_closed_form_causal_rows():
    # Row r of the causal workload keeps columns 0..r mod 4096: row 0 has a
    # single finite entry, so its softmax is exactly one-hot; every masked
    # entry is exactly 0.
    w = W.WORKLOADS["causal_32768x4096"]
    x = W.make_input(w, rows=5)
    v = oracle.widen_bf16_bits(W.to_bits_numpy(x))
    y = oracle.softmax_f64(v)
    assert y[0, 0] == 1.0 and np.all(y[0, 1:] == 0.0)
    for r in range(5):
        assert np.all(y[r, r + 1:] == 0.0)
        assert abs(y[r, : r + 1].sum() - 1.0) < 1e-15


def test_spike_rows_ratio():
    # One +50 per row: the ratio y_i / y_j equals exp(x_i - x_j).
    w = W.WORKLOADS["large_1024x262144"]
    x = W.make_input(w, rows=2)
    v = oracle.widen_f32(W.to_bits_numpy(x))
    y = oracle.softmax_f64(v, threads=2)
    for r in range(2):
        i = int(np.argmax(v[r]))
        assert v[r, i] == 50.0
        j = (i + 1) % v.shape[1]
        assert abs(y[r, j] / y[r, i] - np.exp(v[r, j] - v[r, i])) <= 1e-14 * np.exp(v[r, j] - v[r, i])
        assert y[r, i] > 1.0 - 1e-15
