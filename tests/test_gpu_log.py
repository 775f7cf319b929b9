"""GPU parity of log-softmax (rowsm_log_softmax) against the fp64 oracle of
the same definition, for every family and form and every dtype pair; special
values, in place, misaligned rows; and the full-size long-row workloads
(sampled rows element by element, every row through properties that hold at
any size).  Tolerance (oracle/compare.py, compare_log): fp32 output within
2e-5 + 2^-22 |v|, bf16 output one bf16 ulp more; NaN and -inf positions
identical.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare_log, widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, PAIRS, family_accepts

pytestmark = pytest.mark.gpu


def oracle_log(x_cpu: torch.Tensor) -> np.ndarray:
    b = W.to_bits_numpy(x_cpu)
    v = oracle.widen_bf16_bits(b) if x_cpu.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return oracle.log_softmax_f64(v.reshape(-1, x_cpu.shape[-1]), threads=4)


def run_log(x_dev, dout, config=None, out=None):
    y = R.log_softmax(x_dev, out_dtype=DT[dout], out=out, config=config)
    torch.cuda.synchronize()
    return y


def assert_log_parity(x_cpu, y_dev, dout, what=""):
    v = oracle_log(x_cpu)
    y = widen_output(W.to_bits_numpy(y_dev), dout).reshape(v.shape)
    res = compare_log(y, v, dout)
    assert res["ok"], f"{what}: {res}"
    return res


GRID = {
    R.SMALL: [1, 3, 8, 31, 64, 65, 200, 256],
    R.MEDIUM: [7, 33, 1000, 1023, 4096, 4097, 16385, 65536, 151936],
    R.LARGE: [1, 1000, 65540, 100003, 262144],
}


def grid_cases():
    for fam, cols_list in GRID.items():
        for din, dout in PAIRS:
            for cols in cols_list:
                for rows in (3, 37):
                    if rows * cols <= 3_000_000:
                        yield fam, din, dout, rows, cols


@pytest.mark.parametrize("fam,din,dout,rows,cols", list(grid_cases()))
def test_log_family_grid(fam, din, dout, rows, cols):
    if not family_accepts(rows, cols, din, dout, fam):
        pytest.skip("family does not take this shape")
    x = W.random_matrix(rows, cols, din, sigma=6.0, seed=rows * 31 + cols)
    y = run_log(x.to(DEV), dout, config=R.RowsmConfig(variant=fam))
    assert_log_parity(x, y, dout, f"log {R.VARIANT_NAMES[fam]} {rows}x{cols} {din}->{dout}")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("form", ["two_pass", "two_pass_1block", "packed", "split_2"])
def test_log_forms(form, din, dout):
    if form == "two_pass":                 # 16 blocks per row
        rows, cols, cfg = 5, 70001, dict(variant=R.LARGE, split_blocks=-1)
    elif form == "two_pass_1block":
        rows, cols, cfg = 5, 70001, dict(variant=R.LARGE, split_blocks=-1, blocks_per_cu=1)
    elif form == "packed":
        if din != "bf16" or dout != "bf16":
            pytest.skip("the packed form holds bf16 -> bf16 rows")
        rows, cols, cfg = 6, 151936, dict(variant=R.MEDIUM, packed=1)
    else:
        rows, cols, cfg = 7, 20000, dict(variant=R.LARGE, split_blocks=2)
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols)
    y = run_log(x.to(DEV), dout, config=R.RowsmConfig(**cfg))
    assert_log_parity(x, y, dout, f"log {form} {din}->{dout}")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("fam", [R.SMALL, R.MEDIUM, R.LARGE])
def test_log_special_values(fam, din, dout):
    cols = {R.SMALL: 48, R.MEDIUM: 1000, R.LARGE: 70000}[fam]
    x = W.random_matrix(9, cols, "f32", sigma=3.0, seed=11)
    x[0, 5] = float("nan")
    x[1, 0] = float("inf")
    x[2, :] = float("-inf")
    x[3, ::3] = float("-inf")           # -inf entries with a finite max -> -inf
    x[4, :] = 2.5                       # constant row: -ln(cols)
    x[5, :] = -1000.0
    x[5, cols // 2] = 0.0               # dominant entry: 0 there, -1000 elsewhere
    x[6, :-1] = float("-inf")           # single finite entry, at the end
    x[7, :] = 3.0e4                     # large |m|: no error proportional to |m|
    x[7, 1] = 3.0e4 - 0.5
    x[8, :] = -3.0e38                   # differences that overflow are -inf
    x[8, 2] = 3.0e38
    x = x.to(DT[din])
    y = run_log(x.to(DEV), dout, config=R.RowsmConfig(variant=fam))
    assert_log_parity(x, y, dout, f"log special {R.VARIANT_NAMES[fam]} {din}->{dout}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("fam,cols", [(R.SMALL, 64), (R.MEDIUM, 4096), (R.LARGE, 80000)])
def test_log_in_place_and_misaligned(fam, cols, dt):
    x = W.random_matrix(9, cols, dt, sigma=5.0, seed=3)
    xd = x.to(DEV)
    run_log(xd, dt, config=R.RowsmConfig(variant=fam), out=xd)
    assert_log_parity(x, xd, dt, f"log in place {R.VARIANT_NAMES[fam]}")
    # a view one element into its storage: single-element accesses (a small
    # row then holds at most 32 elements)
    mc = 24 if fam == R.SMALL else cols
    base = W.random_matrix(1, 5 * mc + 1, dt, sigma=2.0, seed=cols).to(DEV)
    xm = base.view(-1)[1:].view(5, mc)
    y = run_log(xm, dt, config=R.RowsmConfig(variant=fam))
    assert_log_parity(xm.cpu(), y, dt, f"log misaligned {R.VARIANT_NAMES[fam]}")


def test_log_empty_and_errors():
    x = torch.empty(0, 16, device=DEV)
    assert run_log(x, "f32").shape == (0, 16)
    # output partially overlapping the input: refused before any launch
    x = torch.zeros(4, 64, device=DEV)
    st = R.rowsm_log_softmax(x.data_ptr(), x.data_ptr() + 4, 4, 64, R.F32, R.F32, 0, None)
    assert st == R.EINVAL


@pytest.mark.parametrize("name", ["vocab_4096x151936", "large_1024x262144"])
def test_log_workload_full_size(name):
    w = W.WORKLOADS[name]
    print(f"log workload {name}: {w.rows}x{w.cols} {w.in_dtype}->{w.out_dtype}", flush=True)
    x = W.make_input(w, device=DEV)
    y = torch.empty(w.rows, w.cols, dtype=DT[w.out_dtype], device=DEV)
    st = R.rowsm_log_softmax(x.data_ptr(), y.data_ptr(), w.rows, w.cols, R.dtype_code(x.dtype),
                             R.dtype_code(y.dtype), torch.cuda.current_stream().cuda_stream,
                             None)
    assert st == R.OK
    torch.cuda.synchronize()
    g = np.random.default_rng(99)
    rows = sorted({0, w.rows - 1, w.rows // 3} | set(int(r) for r in g.integers(0, w.rows, 6)))
    assert_log_parity(x[rows].cpu(), y[rows].cpu(), w.out_dtype, f"log {name} rows {rows}")
    # every row: finite, <= 0 and sum exp(y) = 1
    for r0 in range(0, w.rows, 256):
        yb = y[r0:r0 + 256].double()
        assert torch.isfinite(yb).all()
        assert float(yb.max()) <= 0.0
        assert float((torch.logsumexp(yb, dim=1)).abs().max()) <= 2e-5
    if w.structure == "outliers":
        # the k row maxima hold -ln k
        for r0 in range(0, w.rows, 512):
            xb = x[r0:r0 + 512].float()
            at_max = xb == xb.max(dim=1, keepdim=True).values
            k = at_max.sum(dim=1, keepdim=True).double()
            want = (-torch.log(k)).expand(-1, w.cols)
            got = y[r0:r0 + 512].double()
            assert float((got - want)[at_max].abs().max()) <= 2e-5 + 2.0 ** -22 * 8
    del x, y
    torch.cuda.empty_cache()


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("rows,cols", [(2, 65536), (24, 151936), (5, 262144)])
def test_log_few_rows_launcher_choice(rows, cols, din, dout):
    x = W.random_matrix(rows, cols, din, sigma=5.0, seed=rows + 7 * cols)
    y = run_log(x.to(DEV), dout)
    assert_log_parity(x, y, dout, f"log few rows {rows}x{cols} {din}->{dout}")


@pytest.mark.parametrize("din,dout", [("bf16", "f32"), ("f32", "f32")])
def test_log_split_prefetch_form(din, dout):
    cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=16, blocks_per_cu=1, prefetch=1)
    x = W.random_matrix(200, 151936, din, sigma=4.0, seed=3)
    y = run_log(x.to(DEV), dout, config=cfg)
    assert_log_parity(x, y, dout, f"log prefetch {din}->{dout}")


def test_log_bounded_writes_and_deterministic():
    for fam, cols in ((R.SMALL, 64), (R.MEDIUM, 4096), (R.LARGE, 151936)):
        rows = max(2, 1_000_000 // cols)
        x = W.random_matrix(rows, cols, "bf16", sigma=6.0, seed=cols).to(DEV)
        x0 = x.clone()
        guard, n = 4096, rows * cols
        buf = torch.full((n + 2 * guard,), -123.0, device=DEV)
        y = buf[guard:guard + n].view(rows, cols)
        run_log(x, "f32", config=R.RowsmConfig(variant=fam), out=y)
        y2 = run_log(x, "f32", config=R.RowsmConfig(variant=fam))
        assert torch.equal(y, y2)
        assert torch.all(buf[:guard] == -123.0) and torch.all(buf[guard + n:] == -123.0)
        assert torch.equal(x, x0)


@pytest.mark.parametrize("cols,din,dout,want", [
    (6144, "f32", "f32", ("large", "split=1 ", "block=512 ")),
    (2560, "bf16", "bf16", ("medium", "wpr=4 ", "block=256 ")),
    (10240, "bf16", "f32", ("large", "split=2 ", "block=256 ")),
    (6656, "f32", "bf16", ("medium", "wpr=8 ", "vpl=4 ")),
    (8192, "f32", "bf16", ("large", "split=1 ", "block=512 "))])
def test_log_measured_launch_shapes(cols, din, dout, want):
    # full launches of medium-length rows take the same measured shapes as
    # softmax; sampled rows element by element
    rows = 8201
    st, desc = R.rowsm_describe_op(R.OP_LOG_SOFTMAX, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    assert st == R.OK and all(w in desc for w in want), desc
    print(f"log measured shape {rows}x{cols} {din}->{dout}: {desc}", flush=True)
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols + 3, device=DEV)
    y = run_log(x, dout)
    sample = list(range(0, rows, 101)) + [rows - 1]
    assert_log_parity(x[sample].cpu(), y[sample].cpu(), dout, f"log {rows}x{cols} [{desc}]")
    del x, y
