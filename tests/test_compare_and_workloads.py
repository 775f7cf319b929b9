"""The parity comparator's tolerance rules and the workload recipes (no GPU)."""
import numpy as np
import torch

from oracle.compare import compare, ulp_bf16, widen_output
from paper_2607_23089_amd import workloads as W


def bf16_bits(values):
    return torch.tensor(values, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy()


def test_ulp_bf16_binades():
    assert ulp_bf16(np.array([1.0]))[0] == 2.0 ** -7
    assert ulp_bf16(np.array([1.5]))[0] == 2.0 ** -7
    assert ulp_bf16(np.array([0.99]))[0] == 2.0 ** -8
    assert ulp_bf16(np.array([2.0 ** -126]))[0] == 2.0 ** -133
    assert ulp_bf16(np.array([2.0 ** -140]))[0] == 2.0 ** -133  # subnormal range
    assert ulp_bf16(np.array([-3.0]))[0] == 2.0 ** -6


def test_f32_rule():
    v = np.array([0.5, 0.25, 0.0, np.nan])
    ok = compare(np.array([0.5 + 1.9e-6, 0.25, 0.0, np.nan]), v, "f32")
    assert ok["ok"]
    assert not compare(np.array([0.5 + 2.1e-6, 0.25, 0.0, np.nan]), v, "f32")["ok"]
    r = compare(np.array([0.5, 0.25, 1e-30, np.nan]), v, "f32")   # zero must stay zero
    assert not r["ok"] and r["zero_mismatch"] == 1
    r = compare(np.array([0.5, 0.25, 0.0, 0.1]), v, "f32")        # NaN pattern
    assert not r["ok"] and r["nan_mismatch"] == 1


def test_bf16_rule_one_ulp():
    v = np.array([0.3, 1.0 - 1e-9, 2.0 ** -130])
    y_good = widen_output(bf16_bits([0.3, 1.0, 0.0]), "bf16")
    assert compare(y_good, v, "bf16")["ok"]          # RNE result, subnormal flushed
    # two bf16 steps away from 0.3 is outside 1 ulp
    y_bad = y_good.copy()
    y_bad[0] = y_good[0] + 2 * 2.0 ** -9
    assert not compare(y_bad, v, "bf16")["ok"]


def test_widen_output_roundtrip():
    vals = [1.0, -2.5, 0.0078125]
    assert np.array_equal(widen_output(bf16_bits(vals), "bf16"), np.array(vals))
    assert np.array_equal(widen_output(np.array(vals, dtype=np.float32), "f32"), vals)


def test_workload_table():
    w = W.WORKLOADS
    assert (w["fp32_64x1000"].rows, w["fp32_64x1000"].cols) == (64, 1000)
    assert w["small_262144x64"].algorithmic_bytes == 67108864
    assert w["causal_32768x4096"].algorithmic_bytes == 536870912
    assert w["large_1024x262144"].algorithmic_bytes == 2147483648
    assert w["vocab_4096x151936"].algorithmic_bytes == 3733979136
    assert W.outlier_count(w["vocab_4096x151936"]) == 622330


def test_recipes_on_cpu():
    c1 = W.make_input(W.WORKLOADS["fp32_64x1000"])
    g = torch.Generator().manual_seed(0)
    assert torch.equal(c1, torch.randn(64, 1000, generator=g))          # N(0,1), seed 0
    causal = W.make_input(W.WORKLOADS["causal_32768x4096"], rows=6)
    assert causal.dtype == torch.bfloat16
    for r in range(6):
        assert torch.isinf(causal[r, r + 1:]).all() and torch.isfinite(causal[r, : r + 1]).all()
    spike = W.make_input(W.WORKLOADS["large_1024x262144"], rows=3)
    assert ((spike == 50.0).sum(dim=1) >= 1).all()
    vocab = W.make_input(W.WORKLOADS["vocab_4096x151936"], rows=2)
    big = vocab.float().abs() == 9984.0
    assert 0 < int(big.sum()) <= 2 * 151936 // 1000 + 1
    # seeds are honoured: same seed, same tensor
    assert torch.equal(W.random_matrix(5, 7, "bf16", 3.0, seed=4),
                       W.random_matrix(5, 7, "bf16", 3.0, seed=4))


def test_log_rule():
    from oracle.compare import compare_log
    v = np.array([0.0, -1.0, -20.0, -np.inf, np.nan, -1e-7])
    assert compare_log(v.copy(), v, "f32")["ok"]
    y = v.copy()
    y[2] = -20.0 - (2e-5 + 2.0 ** -22 * 20) * 1.01      # just over the bound
    r = compare_log(y, v, "f32")
    assert not r["ok"] and r["n_over_tol"] == 1
    y = v.copy()
    y[1] = -np.inf                                       # -inf where v is finite
    assert compare_log(y, v, "f32")["inf_mismatch"] == 1
    y = v.copy()
    y[3] = -1e30                                         # finite where v is -inf
    assert not compare_log(y, v, "f32")["ok"]
    y = v.copy()
    y[0] = np.nan
    assert compare_log(y, v, "f32")["nan_mismatch"] == 1
    # bf16: one ulp of v on top of the fp32 bound
    y = v.copy()
    y[2] = -20.0 - 2.0 ** -3                              # ulp_bf16(20) = 2^-3
    assert compare_log(y, v, "bf16")["ok"]
    y[2] = -20.0 - 2.0 ** -2
    assert not compare_log(y, v, "bf16")["ok"]
    # a finite v beyond the output range must come out as -inf
    w = np.array([-6e38])
    assert compare_log(np.array([-np.inf]), w, "f32")["ok"]
    assert not compare_log(np.array([-3.4e38]), w, "f32")["ok"]


def test_backward_rule():
    from oracle.compare import compare_backward
    import oracle
    rng = np.random.default_rng(4)
    y = rng.dirichlet(np.full(50, 0.3), size=6)
    dy = rng.normal(size=(6, 50))
    y[2, 7] = 0.0
    v = oracle.softmax_backward_f64(y, dy)
    assert compare_backward(v.copy(), v, y, dy, "f32")["ok"]
    # fp32 evaluation of the same formula is inside the bound
    y32, dy32 = y.astype(np.float32), dy.astype(np.float32)
    d32 = np.sum(y32 * dy32, axis=1, keepdims=True, dtype=np.float32)
    g32 = (y32 * (dy32 - d32)).astype(np.float64)
    v32 = oracle.softmax_backward_f64(y32.astype(np.float64), dy32.astype(np.float64))
    assert compare_backward(g32, v32, y32, dy32, "f32")["ok"]
    # a dropped product in the dot is far outside it
    bad = v.copy()
    k = int(np.argmax(np.abs(y[1] * dy[1])))
    bad[1] = y[1] * (dy[1] - (np.sum(y[1] * dy[1]) - y[1, k] * dy[1, k]))
    assert not compare_backward(bad, v, y, dy, "f32")["ok"]
    # y == 0 must give exact zeros; NaN positions must agree
    bad = v.copy()
    bad[2, 7] = 1e-30
    assert compare_backward(bad, v, y, dy, "f32")["zero_mismatch"] == 1
    bad = v.copy()
    bad[0, 0] = np.nan
    assert compare_backward(bad, v, y, dy, "f32")["nan_mismatch"] == 1


def test_backward_inputs_are_probability_rows():
    from paper_2607_23089_amd import workloads as W
    w = W.BACKWARD_WORKLOADS["bwd_causal_32768x4096"]
    y, dy = W.make_backward_inputs(w, rows=6)
    yf = y.float()
    assert y.dtype == torch.bfloat16 and dy.shape == y.shape
    assert torch.all(yf >= 0)
    assert float((yf.sum(1) - 1).abs().max()) < 0.02          # bf16-rounded rows
    for r in range(6):
        assert torch.all(yf[r, r + 1:] == 0)                   # causal zeros
    y2, _ = W.make_backward_inputs(w, rows=6)
    assert torch.equal(y, y2)                                   # seeded
