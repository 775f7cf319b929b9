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
