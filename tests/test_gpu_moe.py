"""GPU parity of the MoE group score (rowsm_moe_group_top2) against the fp64
oracle: bit-exact (the result is one fp32 addition of two stored values,
rounded to the output dtype; +0 and -0 compare equal), NaN positions
identical.  Every group size, dtype pair, vector width and groups-per-lane
setting; ties, special values, ragged group counts, misaligned scores,
errors; and the full-size workloads (sampled tokens against the oracle,
every group against torch.topk).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, PAIRS

pytestmark = pytest.mark.gpu


def widen_in(t: torch.Tensor) -> np.ndarray:
    b = W.to_bits_numpy(t)
    v = oracle.widen_bf16_bits(b) if t.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return v.reshape(-1, t.shape[-1])


def assert_moe_exact(scores_cpu, out_dev, group, dout, what=""):
    v = oracle.moe_group_top2_f64(widen_in(scores_cpu), group, dout)
    got = widen_output(W.to_bits_numpy(out_dev), dout).reshape(v.shape)
    nan_ok = np.array_equal(np.isnan(got), np.isnan(v))
    eq = (got == v) | np.isnan(v)
    assert nan_ok and eq.all(), (
        f"{what}: {int((~eq).sum())} of {v.size} differ; first at "
        f"{np.argwhere(~eq)[:3].tolist()} got {got[~eq][:3]} want {v[~eq][:3]}")


def run_moe(scores_dev, group, dout, config=None, out=None):
    o = R.moe_group_top2(scores_dev, group, out_dtype=DT[dout], out=out, config=config)
    torch.cuda.synchronize()
    return o


def tie_heavy(tokens, experts, dtype, seed):
    """Scores drawn from 8 values: most groups hold tied maxima."""
    g = torch.Generator().manual_seed(seed)
    return (torch.randint(0, 8, (tokens, experts), generator=g).float() * 0.25 - 1.0).to(DT[dtype])


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("group", [2, 4, 8, 16, 32, 64])
@pytest.mark.parametrize("rpl", [0, 1, 2, 8])
def test_moe_grid(group, din, dout, rpl):
    cfg = R.RowsmConfig(rows_per_lane=rpl) if rpl else None
    for tokens, experts in ((1, group), (37, 4 * group), (1000, 256 if group <= 256 else group)):
        x = W.random_matrix(tokens, experts, din, sigma=1.0, seed=tokens + group)
        o = run_moe(x.to(DEV), group, dout, config=cfg)
        assert_moe_exact(x, o, group, dout, f"{tokens}x{experts} G={group} {din}->{dout} rpl={rpl}")
        xt = tie_heavy(tokens, experts, din, seed=group)
        o = run_moe(xt.to(DEV), group, dout, config=cfg)
        assert_moe_exact(xt, o, group, dout, f"ties {tokens}x{experts} G={group} {din}->{dout}")


@pytest.mark.parametrize("din", ["f32", "bf16"])
@pytest.mark.parametrize("vw", [1, 2, 4, 8])
def test_moe_vector_widths(din, vw):
    ib = 4 if din == "f32" else 2
    if vw * ib > 16 or (vw > 1 and vw * ib < 8):
        pytest.skip("width not compiled for this dtype")
    x = tie_heavy(333, 256, din, seed=vw)
    o = run_moe(x.to(DEV), 32, "f32", config=R.RowsmConfig(vw=vw))
    assert_moe_exact(x, o, 32, "f32", f"vw={vw} {din}")


@pytest.mark.parametrize("block,rpl,bpc", [(64, 1, 0), (128, 2, 1), (64, 8, 1)])
def test_moe_block_sizes(block, rpl, bpc):
    # smaller blocks (and a capped grid whose waves stride) give the same
    # bit-exact scores
    x = tie_heavy(4099, 256, "f32", seed=block + rpl)
    o = run_moe(x.to(DEV), 32, "f32",
                config=R.RowsmConfig(block=block, rows_per_lane=rpl, blocks_per_cu=bpc))
    assert_moe_exact(x, o, 32, "f32", f"block={block} rpl={rpl} bpc={bpc}")


@pytest.mark.parametrize("din,dout", PAIRS)
def test_moe_special_values(din, dout):
    x = W.random_matrix(8, 64, "f32", sigma=1.0, seed=3)
    x[0, 5] = float("nan")                       # NaN in group 0 only
    x[1, :32] = float("-inf")                    # all -inf group
    x[2, 0] = float("inf")                       # +inf + finite
    x[2, 1:32] = float("-inf")
    x[2, 1] = 1.0
    x[3, 32] = float("inf")
    x[3, 33:] = float("-inf")                    # +inf + -inf = NaN
    x[4, :32] = 3.0                              # constant group: 6
    x[5, 40] = 1e30
    x[5, 41] = 1e30                              # tied huge maximum
    x[6, :] = -0.0
    x[6, 7] = 0.0                                # signed zeros
    x[7, 10] = 3.0e38
    x[7, 11] = 3.0e38                            # the float sum overflows to +inf
    x = x.to(DT[din])
    o = run_moe(x.to(DEV), 32, dout)
    assert_moe_exact(x, o, 32, dout, f"special {din}->{dout}")
    oc = o.float().cpu()
    assert torch.isnan(oc[0, 0]) and not torch.isnan(oc[0, 1])
    assert oc[1, 0] == float("-inf") and torch.isnan(oc[3, 1]) and oc[4, 0] == 6.0


@pytest.mark.parametrize("din", ["f32", "bf16"])
def test_moe_grid_stride(din):
    # one block per compute unit: every wave strides over many tasks
    x = tie_heavy(100000, 256, din, seed=17)
    o = run_moe(x.to(DEV), 32, "f32", config=R.RowsmConfig(blocks_per_cu=1, rows_per_lane=2))
    assert_moe_exact(x, o, 32, "f32", f"grid stride {din}")


def test_moe_misaligned_and_errors():
    base = tie_heavy(1, 64 * 300 + 1, "bf16", seed=9).to(DEV)
    x = base.view(-1)[1:].view(300, 64)          # 2-byte aligned only
    o = run_moe(x, 32, "f32")
    assert_moe_exact(x.cpu(), o, 32, "f32", "misaligned")
    s = torch.zeros(4, 64, device=DEV)
    out = torch.zeros(4, 2, device=DEV)
    f = R.rowsm_moe_group_top2
    assert f(s.data_ptr(), out.data_ptr(), 4, 64, 24, R.F32, R.F32, 0) == R.EINVAL  # not 2^k
    assert f(s.data_ptr(), out.data_ptr(), 4, 64, 128, R.F32, R.F32, 0) == R.EINVAL
    assert f(s.data_ptr(), out.data_ptr(), 4, 60, 32, R.F32, R.F32, 0) == R.EINVAL  # no divide
    assert f(s.data_ptr(), s.data_ptr() + 64, 4, 64, 32, R.F32, R.F32, 0) == R.EINVAL
    assert f(s.data_ptr(), out.data_ptr() + 2, 4, 64, 32, R.F32, R.F32, 0) == R.EINVAL
    assert f(s.data_ptr(), out.data_ptr(), 0, 64, 32, R.F32, R.F32, 0) == R.OK
    assert run_moe(torch.empty(0, 64, device=DEV), 32, "f32").shape == (0, 2)


@pytest.mark.parametrize("name", list(W.MOE_WORKLOADS))
def test_moe_workload_full_size(name):
    w = W.MOE_WORKLOADS[name]
    print(f"moe workload {name}: {w.tokens}x{w.experts} G={w.group} {w.in_dtype}->{w.out_dtype}",
          flush=True)
    x = W.make_moe_scores(w, device=DEV)
    o = torch.empty(w.tokens, w.experts // w.group, dtype=DT[w.out_dtype], device=DEV)
    st = R.rowsm_moe_group_top2(x.data_ptr(), o.data_ptr(), w.tokens, w.experts, w.group,
                                R.dtype_code(x.dtype), R.dtype_code(o.dtype),
                                torch.cuda.current_stream().cuda_stream)
    assert st == R.OK
    torch.cuda.synchronize()
    g = np.random.default_rng(5)
    toks = sorted({0, w.tokens - 1} | set(int(t) for t in g.integers(0, w.tokens, 64)))
    assert_moe_exact(x[toks].cpu(), o[toks].cpu(), w.group, w.out_dtype, f"{name} tokens {toks[:5]}")
    # every group: the fp32 sum of torch.topk's two values
    for t0 in range(0, w.tokens, 1 << 16):
        xb = x[t0:t0 + (1 << 16)].float().view(-1, w.experts // w.group, w.group)
        want = torch.topk(xb, 2, dim=-1).values.sum(-1)
        assert torch.equal(o[t0:t0 + (1 << 16)].float(), want)
    del x, o
    torch.cuda.empty_cache()


def test_moe_bounded_writes_and_scores_untouched():
    x = W.random_matrix(3333, 256, "bf16", seed=8).to(DEV)
    x0 = x.clone()
    guard, n = 1024, 3333 * 8
    buf = torch.full((n + 2 * guard,), -123.0, device=DEV)
    o = buf[guard:guard + n].view(3333, 8)
    run_moe(x, 32, "f32", out=o)
    assert torch.all(buf[:guard] == -123.0) and torch.all(buf[guard + n:] == -123.0)
    assert torch.equal(x, x0)
    o2 = run_moe(x, 32, "f32")
    assert torch.equal(o, o2)
    assert_moe_exact(x.cpu(), o, 32, "f32", "bounded")
