"""GPU parity of the softmax backward (rowsm_softmax_backward) against the
fp64 oracle of dx = y * (dy - sum(y * dy)), for every family and form and
every dtype pair; special values, in place, misaligned rows, determinism;
and the full-size backward workloads (sampled rows element by element, every
row through properties that hold at any size).  Tolerance (oracle/compare.py,
compare_backward): |dx - v| <= |y| (2^-17 sum|y dy| + 2^-23 |dy - d|) +
2^-23 |v|, one bf16 ulp more for bf16 output; NaN and infinity positions
identical, y == 0 gives exactly 0.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare_backward, widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, PAIRS

pytestmark = pytest.mark.gpu


def widen_in(t: torch.Tensor) -> np.ndarray:
    b = W.to_bits_numpy(t)
    v = oracle.widen_bf16_bits(b) if t.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return v.reshape(-1, t.shape[-1])


def assert_bwd_parity(y_cpu, dy_cpu, dx_dev, dout, what=""):
    y, dy = widen_in(y_cpu), widen_in(dy_cpu)
    v = oracle.softmax_backward_f64(y, dy, threads=4)
    dx = widen_output(W.to_bits_numpy(dx_dev), dout).reshape(v.shape)
    res = compare_backward(dx, v, y, dy, dout)
    assert res["ok"], f"{what}: {res}"
    return res


def run_bwd(y_dev, dy_dev, dout, config=None, out=None):
    dx = R.softmax_backward(y_dev, dy_dev, out_dtype=DT[dout], out=out, config=config)
    torch.cuda.synchronize()
    return dx


def bwd_accepts(rows, cols, din, dout, cfg):
    st, _ = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, R.dtype_code(DT[din]),
                                R.dtype_code(DT[dout]), cfg)
    return st == R.OK


def inputs(rows, cols, din, alpha=0.3, seed=0):
    y = W.random_probabilities(rows, cols, din, alpha, seed=seed + 2)
    dy = W.random_matrix(rows, cols, din, sigma=1.0, seed=seed + 3)
    return y, dy


GRID = {
    R.SMALL: [1, 2, 7, 8, 31, 64, 65, 200, 256],
    R.MEDIUM: [1, 33, 1000, 1023, 4096, 4097, 16385, 32768, 65536],
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
def test_bwd_family_grid(fam, din, dout, rows, cols):
    cfg = R.RowsmConfig(variant=fam)
    if not bwd_accepts(rows, cols, din, dout, cfg):
        pytest.skip("family does not take this shape")
    y, dy = inputs(rows, cols, din, seed=rows + cols)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout, config=cfg)
    assert_bwd_parity(y, dy, dx, dout, f"bwd {R.VARIANT_NAMES[fam]} {rows}x{cols} {din}->{dout}")


FORMS = {
    "two_pass": (5, 70001, dict(variant=R.LARGE, split_blocks=-1)),      # 16 blocks per row
    "two_pass_1block": (5, 70001, dict(variant=R.LARGE, split_blocks=-1, blocks_per_cu=1)),
    "two_pass_long": (2, (1 << 21) + 5, dict(variant=R.LARGE)),         # past the split form
    "two_pass_u8": (3, 150001, dict(variant=R.LARGE, split_blocks=-1, tile_vectors=8)),
    "split_2": (7, 20000, dict(variant=R.LARGE, split_blocks=2)),
    "split_64": (3, 300000, dict(variant=R.LARGE, split_blocks=64)),
    "split_1024": (4, 200000, dict(variant=R.LARGE, block=1024)),
    "medium_wpr16": (9, 3000, dict(variant=R.MEDIUM, waves_per_row=16)),
    "medium_rpb1": (9, 3000, dict(variant=R.MEDIUM, waves_per_row=2, rows_per_block=1)),
    "small_rpl1": (100, 40, dict(variant=R.SMALL, rows_per_lane=1)),
    "small_rpl8_l32": (100, 40, dict(variant=R.SMALL, rows_per_lane=8, lanes_per_row=32)),
}


@pytest.mark.parametrize("rows,cols,din,dout,want", [
    (1024, 8192, "f32", "f32", ("wpr=4 ", "vpl=8 ")),
    (2048, 6144, "bf16", "f32", ("wpr=2 ", "vpl=12 ")),
    (1531, 16384, "bf16", "bf16", ("wpr=4 ", "vpl=8 "))])
def test_bwd_few_rows_per_cu_shapes(rows, cols, din, dout, want):
    # launches of 4-16 rows per compute unit: few waves per row, many bytes of
    # each input per lane; sampled rows against the oracle
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("medium") and all(w in desc for w in want), desc
    y, dy = inputs(rows, cols, din, alpha=0.2, seed=rows)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout)
    sample = list(range(0, rows, 11)) + [rows - 1]
    assert_bwd_parity(y[sample], dy[sample], dx[sample].cpu(), dout,
                      f"bwd {rows}x{cols} {din}->{dout} [{desc}]")


BWD_MEASURED_SHAPES = [  # (cols, din, dout, expected plan fields): one length per table entry
    (1200, "bf16", "bf16", ("medium", "wpr=2 ", "block=128 ")),
    (2000, "bf16", "bf16", ("medium", "wpr=4 ", "block=256 ")),
    (2800, "bf16", "bf16", ("large", "split=1 ", "block=256 ")),
    (4800, "bf16", "bf16", ("medium", "wpr=8 ", "block=512 ")),
    (8000, "bf16", "bf16", ("large", "split=1 ", "block=512 ")),
    (12000, "bf16", "bf16", ("medium", "wpr=16 ", "block=1024 ")),
    (16000, "bf16", "bf16", ("large", "split=2 ", "block=256 ")),
    (24000, "bf16", "bf16", ("large", "split=2 ", "block=512 ")),
    (32000, "bf16", "bf16", ("large", "split=4 ", "block=256 ")),
    (800, "f32", "f32", ("medium", "wpr=4 ", "block=256 ")),
    (1680, "f32", "f32", ("large", "split=1 ", "block=256 ")),
    (2400, "f32", "f32", ("medium", "wpr=8 ", "block=512 ")),
    (4000, "f32", "f32", ("large", "split=1 ", "block=512 ")),
    (8000, "f32", "f32", ("large", "split=2 ", "block=256 ")),
    (16384, "f32", "f32", ("large", "split=2 ", "block=512 ")),
    (600, "bf16", "f32", ("medium", "wpr=2 ", "block=128 ")),
    (1200, "bf16", "f32", ("medium", "wpr=4 ", "block=256 ")),
    (2400, "bf16", "f32", ("medium", "wpr=4 ", "block=512 ")),
    (4000, "bf16", "f32", ("medium", "wpr=8 ", "block=512 ")),
    (8000, "bf16", "f32", ("medium", "wpr=4 ", "nv=8 ", "block=256 ")),
    (12000, "bf16", "f32", ("medium", "wpr=16 ", "block=1024 ")),
    (600, "f32", "bf16", ("medium", "wpr=2 ", "block=256 ")),
    (1024, "f32", "bf16", ("medium", "wpr=4 ", "block=256 ")),
    (1680, "f32", "bf16", ("large", "split=1 ", "block=256 ")),
    (2400, "f32", "bf16", ("medium", "wpr=8 ", "block=512 ")),
    (4000, "f32", "bf16", ("large", "split=1 ", "block=512 ")),
    (5200, "f32", "bf16", ("medium", "wpr=8 ", "block=1024 ")),
    (8000, "f32", "bf16", ("large", "split=2 ", "block=256 ")),
    (12000, "f32", "bf16", ("large", "split=2 ", "block=512 ")),
]


@pytest.mark.parametrize("cols,din,dout,want", BWD_MEASURED_SHAPES)
def test_bwd_measured_launch_shapes(cols, din, dout, want):
    # full launches (8201 rows: >= 32 per compute unit, ragged) take the
    # measured backward shapes; sampled rows, the last ones among them,
    # against the oracle
    rows = 8201
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith(want[0]) and all(w in desc for w in want), desc
    print(f"bwd measured shape {rows}x{cols} {din}->{dout}: {desc}", flush=True)
    y = W.random_probabilities(rows, cols, din, 0.3, seed=cols + 2, device=DEV)
    dy = W.random_matrix(rows, cols, din, sigma=1.0, seed=cols + 3, device=DEV)
    dx = run_bwd(y, dy, dout)
    sample = list(range(0, rows, 131)) + [rows - 2, rows - 1]
    assert_bwd_parity(y[sample].cpu(), dy[sample].cpu(), dx[sample].cpu(), dout,
                      f"bwd {rows}x{cols} {din}->{dout} [{desc}]")
    del y, dy, dx


@pytest.mark.parametrize("cols,dt", [(4000, "f32"), (16000, "bf16")])
def test_bwd_in_place_full_launch(cols, dt):
    # in place, a full launch whose measured shape is the single-read form
    # keeps the medium form (no exchanging form in place): over dy and over y
    rows = 8201
    y = W.random_probabilities(rows, cols, dt, 0.3, seed=cols, device=DEV)
    dy = W.random_matrix(rows, cols, dt, sigma=1.0, seed=cols + 1, device=DEV)
    sample = list(range(0, rows, 257)) + [rows - 1]
    ys, dys = y[sample].cpu(), dy[sample].cpu()
    for over in ("dy", "y"):
        yd, dyd = y.clone(), dy.clone()
        out = dyd if over == "dy" else yd
        run_bwd(yd, dyd, dt, out=out)
        assert_bwd_parity(ys, dys, out[sample].cpu(), dt, f"bwd in place over {over} {rows}x{cols}")
        del yd, dyd


@pytest.mark.parametrize("rows,cols,din,dout", [
    (262144, 64, "bf16", "bf16"), (262147, 64, "bf16", "bf16"), (131072, 128, "f32", "f32"),
    (1048576, 32, "bf16", "f32"), (786435, 16, "f32", "bf16")])
def test_bwd_small_one_wave_blocks(rows, cols, din, dout):
    # launches of at least 96 MiB of rows that fill their lanes: one-wave
    # blocks, one row group per lane (ragged row counts included); sampled
    # rows, the last ones among them, against the oracle
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("small") and "block=64 " in desc and "rpl=1 " in desc
    y, dy = inputs(rows, cols, din, alpha=0.3, seed=rows + cols)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout)
    sample = list(range(0, rows, 997)) + list(range(rows - 9, rows))
    assert_bwd_parity(y[sample], dy[sample], dx[sample].cpu(), dout,
                      f"bwd {rows}x{cols} {din}->{dout} [{desc}]")


@pytest.mark.parametrize("rows,cols,din,dout", [
    (1024, 16384, "f32", "f32"), (1024, 32768, "bf16", "f32"), (1024, 32768, "bf16", "bf16"),
    (300, 65536, "f32", "f32"), (16, 16384, "f32", "f32"), (48, 49152, "bf16", "f32"),
    (127, 32768, "bf16", "bf16"), (100, 16384, "f32", "bf16")])
def test_bwd_wide_rows_take_split_form(rows, cols, din, dout):
    # rows that would need all 16 waves of one block, many rows or fewer
    # than cus / 2: the split form (the launcher's own choice)
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("large") and "split=0" not in desc, desc
    y, dy = inputs(rows, cols, din, alpha=0.1, seed=rows + cols)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout)
    assert_bwd_parity(y, dy, dx, dout, f"bwd wide rows {rows}x{cols} {din}->{dout} [{desc}]")


@pytest.mark.parametrize("rows,cols,din,dout", [
    (204600, 131, "bf16", "bf16"), (153450, 132, "bf16", "f32"), (122760, 90, "f32", "bf16"),
    (291271, 90, "f32", "f32"), (349525, 150, "bf16", "bf16"), (81707, 94, "f32", "f32"),
    (288070, 182, "bf16", "bf16"), (163840, 320, "bf16", "bf16")])
def test_bwd_short_rows_looping_grid(rows, cols, din, dout):
    # rows of one wave and one to four slots (parts of 128-byte lines, and
    # whole lines: 640-byte bf16 rows):
    # a grid of about 24 KiB of the three streams per block, whose waves loop
    # over the rows; the output prefilled with NaN so that every row is seen
    # written, sampled rows (the last ones among them) against the oracle
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("medium") and "wpr=1 " in desc, desc
    per_row = cols * (2 * DT[din].itemsize + DT[dout].itemsize)
    grid = max(1024, (-(-rows // max(1, 24576 // per_row)) + 512) // 1024 * 1024)
    assert f"block=512 grid={grid} " in desc, desc
    y, dy = inputs(rows, cols, din, alpha=0.3, seed=rows)
    out = torch.full((rows, cols), float("nan"), dtype=DT[dout], device=DEV)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout, out=out)
    assert bool(torch.isfinite(dx).all())
    sample = list(range(0, rows, 991)) + list(range(rows - 9, rows))
    assert_bwd_parity(y[sample], dy[sample], dx[sample].cpu(), dout,
                      f"bwd short {rows}x{cols} {din}->{dout} [{desc}]")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("form", sorted(FORMS))
def test_bwd_forms(form, din, dout):
    rows, cols, cfg = FORMS[form]
    cfg = R.RowsmConfig(**cfg)
    if not bwd_accepts(rows, cols, din, dout, cfg):
        pytest.skip("form does not take this shape")
    y, dy = inputs(rows, cols, din, alpha=0.1, seed=cols)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout, config=cfg)
    assert_bwd_parity(y, dy, dx, dout, f"bwd {form} {din}->{dout}")


TWO_PASS = -1    # the two-pass LARGE form, several blocks per row
TWO_PASS_1 = -2  # the two-pass LARGE form, one block per row


def special_config(fam):
    if fam == TWO_PASS:
        return R.RowsmConfig(variant=R.LARGE, split_blocks=-1)
    if fam == TWO_PASS_1:
        return R.RowsmConfig(variant=R.LARGE, split_blocks=-1, blocks_per_cu=1)
    return R.RowsmConfig(variant=fam)


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("fam", [R.SMALL, R.MEDIUM, R.LARGE, TWO_PASS, TWO_PASS_1])
def test_bwd_special_values(fam, din, dout):
    cols = {R.SMALL: 48, R.MEDIUM: 1000}.get(fam, 70000)
    y, dy = inputs(8, cols, "f32", seed=5)
    dy[0, 3] = float("nan")              # NaN gradient: the whole row is NaN
    dy[1, 0] = float("inf")              # infinite gradient: d = +inf
    y[2, :] = 0.0                        # zero row: exact zeros
    y[3, ::2] = 0.0                      # zeros inside a row stay exact zeros
    dy[4, :] = 0.75                      # constant gradient: dx ~ 0
    y[5, :] = 0.0
    y[5, cols // 3] = 1.0                # one-hot y: dx = 0 everywhere
    dy[6, :] = 0.0                       # zero gradient
    y[7, 1] = float("nan")               # NaN probability
    y, dy = y.to(DT[din]), dy.to(DT[din])
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout, config=special_config(fam))
    assert_bwd_parity(y, dy, dx, dout, f"bwd special {fam} {din}->{dout}")
    dxc = dx.cpu().float()
    assert torch.isnan(dxc[0]).all()
    # d = +inf: dx = y * (dy - inf) = -inf where y > 0, NaN at the inf entry
    # (inf - inf) and where y == 0 (0 * -inf)
    yc = y.float()
    assert torch.isnan(dxc[1, 0])
    assert torch.all(dxc[1, 1:][yc[1, 1:] > 0] == float("-inf"))
    assert torch.isnan(dxc[1, 1:][yc[1, 1:] == 0]).all()
    assert torch.all(dxc[2] == 0) and torch.all(dxc[5] == 0) and torch.all(dxc[6] == 0)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("fam,cols", [(R.SMALL, 64), (R.MEDIUM, 4096), (R.LARGE, 80000)])
def test_bwd_in_place(fam, cols, dt):
    cfg = R.RowsmConfig(variant=fam)
    y, dy = inputs(9, cols, dt, seed=9)
    yd, dyd = y.to(DEV), dy.to(DEV)
    run_bwd(yd, dyd, dt, config=cfg, out=dyd)          # dx over dy
    assert_bwd_parity(y, dy, dyd, dt, f"bwd in place over dy {R.VARIANT_NAMES[fam]}")
    yd, dyd = y.to(DEV), dy.to(DEV)
    run_bwd(yd, dyd, dt, config=cfg, out=yd)           # dx over y
    assert_bwd_parity(y, dy, yd, dt, f"bwd in place over y {R.VARIANT_NAMES[fam]}")


@pytest.mark.parametrize("din,dout", PAIRS)
def test_bwd_misaligned_rows(din, dout):
    for fam, cols in ((R.SMALL, 24), (R.MEDIUM, 1024), (R.LARGE, 65600)):
        yb, dyb = inputs(1, 5 * cols + 1, din, seed=cols)
        y = yb.to(DEV).view(-1)[1:].view(5, cols)
        dy = dyb.to(DEV).view(-1)[1:].view(5, cols)
        dx = run_bwd(y, dy, dout, config=R.RowsmConfig(variant=fam))
        assert_bwd_parity(y.cpu(), dy.cpu(), dx, dout,
                          f"bwd misaligned {R.VARIANT_NAMES[fam]} {din}->{dout}")


def test_bwd_same_buffer_inputs_and_errors():
    # y and dy may be the same buffer (read only)
    y, _ = inputs(6, 3000, "f32", seed=1)
    yd = y.to(DEV)
    dx = run_bwd(yd, yd, "f32")
    assert_bwd_parity(y, y, dx, "f32", "bwd y == dy")
    # dx partially overlapping an input, or in place with a dtype change:
    # refused before any launch
    yb = torch.zeros(4, 64, device=DEV, dtype=torch.bfloat16)
    d = torch.zeros(4, 64, device=DEV, dtype=torch.bfloat16)
    f = R.rowsm_softmax_backward
    assert f(yb.data_ptr(), d.data_ptr(), yb.data_ptr() + 2, 4, 64, R.BF16, R.BF16, 0) == R.EINVAL
    assert f(yb.data_ptr(), d.data_ptr(), d.data_ptr() + 2, 4, 64, R.BF16, R.BF16, 0) == R.EINVAL
    assert f(yb.data_ptr(), d.data_ptr(), d.data_ptr(), 4, 64, R.BF16, R.F32, 0) == R.EINVAL
    empty = torch.empty(0, 8, device=DEV)
    assert run_bwd(empty, empty, "f32").shape == (0, 8)


def test_bwd_deterministic():
    for fam, cols in ((R.MEDIUM, 8000), (R.LARGE, 150000)):
        y, dy = inputs(16, cols, "f32", seed=2)
        yd, dyd = y.to(DEV), dy.to(DEV)
        a = run_bwd(yd, dyd, "f32", config=R.RowsmConfig(variant=fam))
        b = run_bwd(yd, dyd, "f32", config=R.RowsmConfig(variant=fam))
        assert torch.equal(a, b)


@pytest.mark.parametrize("name", list(W.BACKWARD_WORKLOADS))
def test_bwd_workload_full_size(name):
    w = W.BACKWARD_WORKLOADS[name]
    print(f"backward workload {name}: {w.rows}x{w.cols} {w.in_dtype}->{w.out_dtype}", flush=True)
    y, dy = W.make_backward_inputs(w, device=DEV)
    dx = torch.empty(w.rows, w.cols, dtype=DT[w.out_dtype], device=DEV)
    st = R.rowsm_softmax_backward(y.data_ptr(), dy.data_ptr(), dx.data_ptr(), w.rows, w.cols,
                                  R.dtype_code(y.dtype), R.dtype_code(dx.dtype),
                                  torch.cuda.current_stream().cuda_stream)
    assert st == R.OK
    torch.cuda.synchronize()
    g = np.random.default_rng(7)
    rows = sorted({0, 1, w.rows // 2, w.rows - 1} | set(int(r) for r in g.integers(0, w.rows, 8)))
    assert_bwd_parity(y[rows].cpu(), dy[rows].cpu(), dx[rows].cpu(), w.out_dtype,
                      f"bwd {name} rows {rows}")
    # every row: finite, exact zeros where y is zero, and
    # sum_j dx_j = d (1 - sum_j y_j), small for probability rows
    for r0 in range(0, w.rows, 4096):
        yb, dyb, dxb = y[r0:r0 + 4096].double(), dy[r0:r0 + 4096].double(), dx[r0:r0 + 4096]
        assert torch.isfinite(dxb).all()
        assert torch.all(dxb[yb == 0] == 0)
        d = (yb * dyb).sum(1)
        want = d * (1 - yb.sum(1))
        got = dxb.double().sum(1)
        scale = (yb * dyb.abs()).sum(1) + (yb * (dyb - d[:, None]).abs()).sum(1)
        ulp = 2.0 ** -8 if w.out_dtype == "bf16" else 2.0 ** -22
        assert float(((got - want).abs() - ulp * scale).max()) <= 1e-6
    del y, dy, dx
    torch.cuda.empty_cache()


def test_bwd_and_forward_split_launches_interleaved_on_streams():
    # Forward and backward single-read launches share the device's exchange
    # workspace; interleaved on two streams they must be ordered and exact,
    # and repeats on the same data bitwise equal.
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    cases = [inputs(9, 70000 + 64 * i, "f32", seed=i) for i in range(3)]
    xs = [W.random_matrix(11, 90000 + 8 * i, "bf16", sigma=3.0, seed=i).to(DEV) for i in range(3)]
    dev_cases = [(y.to(DEV), dy.to(DEV)) for y, dy in cases]
    outs = []
    for it in range(12):
        s = s1 if it % 2 == 0 else s2
        k = it % 3
        with torch.cuda.stream(s):
            if (it // 3) % 2 == 0:
                yd, dyd = dev_cases[k]
                outs.append(("bwd", k, R.softmax_backward(yd, dyd, stream=s,
                                                          config=R.RowsmConfig(variant=R.LARGE))))
            else:
                outs.append(("fwd", k, R.softmax(xs[k], out_dtype=torch.float32, variant=R.LARGE,
                                                 stream=s)))
    torch.cuda.synchronize()
    first = {}
    for kind, k, o in outs:
        if (kind, k) not in first:
            first[(kind, k)] = o
            if kind == "bwd":
                assert_bwd_parity(cases[k][0], cases[k][1], o, "f32", f"interleaved bwd {k}")
            else:
                from test_gpu_parity import assert_parity
                assert_parity(xs[k].cpu(), o, "f32", f"interleaved fwd {k}")
        else:
            assert torch.equal(o, first[(kind, k)])


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("rows,cols", [(1, 65536), (8, 65536), (32, 151936), (3, 262144),
                                       (16, 262144)])
def test_bwd_few_rows_launcher_choice(rows, cols, din, dout):
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    assert st == R.OK
    y, dy = inputs(rows, cols, din, alpha=0.2, seed=rows + cols)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout)
    assert_bwd_parity(y, dy, dx, dout, f"bwd few rows {rows}x{cols} {din}->{dout} [{desc}]")


def test_bwd_bounded_writes_and_inputs_untouched():
    # nothing written outside dx; y and dy unchanged
    for fam, cols in ((R.SMALL, 64), (R.MEDIUM, 4096), (R.LARGE, 151936)):
        rows = max(2, 1_000_000 // cols)
        y, dy = inputs(rows, cols, "bf16", seed=cols)
        yd, dyd = y.to(DEV), dy.to(DEV)
        y0, dy0 = yd.clone(), dyd.clone()
        guard, n = 4096, rows * cols
        buf = torch.full((n + 2 * guard,), -123.0, device=DEV)
        dx = buf[guard:guard + n].view(rows, cols)
        run_bwd(yd, dyd, "f32", config=R.RowsmConfig(variant=fam), out=dx)
        assert torch.all(buf[:guard] == -123.0) and torch.all(buf[guard + n:] == -123.0)
        assert torch.equal(yd, y0) and torch.equal(dyd, dy0)
        assert_bwd_parity(y, dy, dx, "f32", f"bounded {R.VARIANT_NAMES[fam]}")
