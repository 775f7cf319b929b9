"""GPU parity of the scaled, causally masked form (rowsm_forward_scaled_causal)
against the fp64 oracle of the same definition, for every family and dtype
pair, plus its identity with the plain form on data that stores the mask.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare, widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, PAIRS

pytestmark = pytest.mark.gpu


def oracle_fused(x_cpu, scale, period, offset, row0=0):
    b = W.to_bits_numpy(x_cpu)
    v = oracle.widen_bf16_bits(b) if x_cpu.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return oracle.softmax_scaled_causal_f64(v, scale, period, offset, threads=4, row0=row0)


def run_fused(x_dev, dout, scale, period, offset, config=None):
    y = R.scaled_causal_softmax(x_dev, scale, period, offset, out_dtype=DT[dout], config=config)
    torch.cuda.synchronize()
    return y


def assert_fused_parity(x_cpu, y_dev, dout, scale, period, offset, what, row0=0):
    v = oracle_fused(x_cpu, scale, period, offset, row0)
    y = widen_output(W.to_bits_numpy(y_dev), dout).reshape(v.shape)
    res = compare(y, v, dout)
    assert res["ok"], f"{what}: {res}"


CASES = [  # (family, cols)
    (R.SMALL, 24), (R.SMALL, 64), (R.SMALL, 200),
    (R.MEDIUM, 1000), (R.MEDIUM, 4096), (R.MEDIUM, 4097),
    (R.LARGE, 40000), (R.LARGE, 151936),
]
MASKS = [(0.125, 0, 0), (1.0, 8, 0), (0.5, 16, 3), (-0.75, 5, -1), (2.0, 3, 1000)]


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("fam,cols", CASES)
def test_fused_grid(fam, cols, din, dout):
    rows = 37 if cols < 100000 else 6
    st, _ = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]), fam)
    if st != R.OK:
        pytest.skip("family does not take this shape")
    x = W.random_matrix(rows, cols, din, sigma=5.0, seed=cols + rows)
    for scale, period, offset in MASKS:
        if period and cols > 1000:
            period, offset = rows, cols - rows     # keys aligned to the end
        cfg = R.RowsmConfig(variant=fam)
        y = run_fused(x.to(DEV), dout, scale, period, offset, config=cfg)
        assert_fused_parity(x, y, dout, scale, period, offset,
                            f"{R.VARIANT_NAMES[fam]} {rows}x{cols} {din}->{dout} "
                            f"scale={scale} period={period} offset={offset}")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("bpc", [0, 1])   # 16 blocks per row, or one
def test_fused_two_pass_form(din, dout, bpc):
    x = W.random_matrix(5, 70001, din, sigma=3.0, seed=7)
    cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=-1, blocks_per_cu=bpc)
    y = run_fused(x.to(DEV), dout, 0.3, 5, 40000, config=cfg)
    assert_fused_parity(x, y, dout, 0.3, 5, 40000, f"two-pass fused bpc={bpc} {din}->{dout}")


def test_fully_masked_rows_are_nan_and_masked_entries_zero():
    x = W.random_matrix(8, 512, "f32", sigma=2.0, seed=1)
    y = run_fused(x.to(DEV), "f32", 1.0, 4, -1).cpu()
    assert torch.isnan(y[0]).all() and torch.isnan(y[4]).all()
    for r in (1, 2, 3, 5, 6, 7):
        q = r % 4
        assert torch.all(y[r, q:] == 0) and torch.all(y[r, :q] > 0)


@pytest.mark.parametrize("fam,cols", [(R.SMALL, 64), (R.MEDIUM, 4096), (R.LARGE, 40000),
                                      (R.LARGE, 70001)])
def test_fused_special_rows(fam, cols):
    # NaN or +inf among the kept columns makes the whole row NaN, masked
    # columns included (0 / NaN); -inf among the kept ones is an ordinary 0.
    x = W.random_matrix(8, cols, "f32", sigma=2.0, seed=2)
    x[1, 0] = float("nan")
    x[2, 1] = float("inf")
    x[3, 0] = float("-inf")
    x[5, 0] = float("nan")     # kept for query 5 % 4 = 1 (columns 0..1)
    cfg = R.RowsmConfig(variant=fam) if cols != 70001 else R.RowsmConfig(variant=fam,
                                                                          split_blocks=-1)
    for din, dout in PAIRS:
        xx = x.to(DT[din])
        y = run_fused(xx.to(DEV), dout, 1.5, 4, 0, config=cfg)
        assert_fused_parity(xx, y, dout, 1.5, 4, 0, f"special {fam} {cols} {din}->{dout}")


def test_causal_workload_in_kernel_mask_matches_stored_mask():
    # The causal workload at full size: softmax with the mask computed in the
    # kernel from the indices (x holds no -inf) must equal, bit for bit, the
    # plain kernel on the same scores with the mask stored as -inf (in the
    # same launch shape, same arithmetic: scale 1 multiplies exactly).
    w = W.WORKLOADS["causal_32768x4096"]
    xm = W.make_input(w, device=DEV)                       # mask stored as -inf
    g = torch.Generator(device=DEV).manual_seed(0)
    x = (torch.randn(w.rows, w.cols, generator=g, device=DEV) * w.sigma).to(torch.bfloat16)
    assert torch.equal(torch.where(torch.isinf(xm), xm, x), xm)
    y_fused = R.scaled_causal_softmax(x, 1.0, w.period, 0)
    # the plain form forced to the fused form's launch shape (2 waves per row,
    # 2 rows per block) sums in the same order
    same_shape = R.RowsmConfig(variant=R.MEDIUM, waves_per_row=2, rows_per_block=2)
    y_plain = R.softmax(xm, config=same_shape)
    torch.cuda.synchronize()
    assert torch.equal(y_plain, y_fused)
    for r in (0, 1, 4095, 4096, 20000, 32767):
        assert_fused_parity(x[r:r + 1].cpu(), y_fused[r:r + 1].cpu(), "bf16", 1.0, w.period, 0,
                            f"fused causal row {r}", row0=r)


@pytest.mark.parametrize("cols,din,want", [
    (1024, "f32", ("medium", "wpr=2 ", "block=128 ")),
    (4096, "f32", ("medium", "wpr=4 ", "vpl=4 ")),
    (12288, "f32", ("medium", "wpr=16 ", "vpl=3 ")),
    (16384, "f32", ("large", "split=2 ", "block=256 ")),
    (2048, "bf16", ("medium", "wpr=2 ", "vpl=4 ", "block=128 ")),
    (5120, "bf16", ("medium", "wpr=4 ", "vpl=5 ")),
    (16384, "bf16", ("large", "split=2 ", "block=256 "))])
def test_fused_measured_launch_shapes(cols, din, want):
    # full launches of causal heads with fp32 output take the measured fused
    # shapes; blocks of sampled rows element by element against the oracle
    rows, scale = 8201, 0.125
    st, desc = R.rowsm_describe_op(R.OP_SCALED_CAUSAL, rows, cols, R.dtype_code(DT[din]), R.F32)
    assert st == R.OK and all(w in desc for w in want), desc
    print(f"fused measured shape {rows}x{cols} {din}->f32: {desc}", flush=True)
    x = W.random_matrix(rows, cols, din, sigma=5.0, seed=cols + 11, device=DEV)
    y = R.scaled_causal_softmax(x, scale, cols, 0, out_dtype=torch.float32)
    torch.cuda.synchronize()
    for r0 in (0, cols - 3, rows // 2, rows - 4):
        xs, ys = x[r0:r0 + 4].cpu(), y[r0:r0 + 4].cpu()
        assert_fused_parity(xs, ys, "f32", scale, cols, 0, f"{rows}x{cols} rows {r0}+ [{desc}]",
                            row0=r0)
    del x, y
