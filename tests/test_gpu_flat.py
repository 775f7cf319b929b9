"""GPU parity of the flat short-row form (rows of a width that is not a
multiple of the 16-byte vector width, up to 1024 columns, read and written as
one stream of whole vectors aligned to the tensor and regrouped into rows
through LDS) against the fp64 oracle: every dtype pair, widths from 1 column
to 1017-1023, row counts that leave a partial final tile and a last vector
reaching past the end of the tensor, softmax and log-softmax, special
values, in place, guard bands before and after the output, and the form
asked for by configuration.
"""
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare_log, widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, PAIRS, assert_parity

pytestmark = pytest.mark.gpu


def full_vw(din, dout):
    return 16 // max(4 if din == "f32" else 2, 4 if dout == "f32" else 2)


def flat_cfg(din, dout):
    # the flat form asked for: the small variant at the full vector width
    return R.RowsmConfig(variant=R.SMALL, vw=full_vw(din, dout))


def describe(rows, cols, din, dout, cfg=None, op=R.OP_SOFTMAX):
    st, desc = R.rowsm_describe_op(op, rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]),
                                   cfg)
    assert st == R.OK, desc
    return desc


WIDTHS = [1, 3, 5, 7, 9, 13, 21, 37, 63, 77, 101, 129, 255, 257, 511, 513, 1001, 1017]


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("cols", WIDTHS)
def test_flat_widths(cols, din, dout):
    # three tiles and a partial fourth; the row count makes the tensor end
    # inside a vector
    vw = full_vw(din, dout)
    if cols % vw == 0:
        pytest.skip("a multiple of the vector width")
    g = (4 * 64 * vw - (vw - 1)) // cols
    rows = 3 * g + max(1, g // 2)
    if (rows * cols) % vw == 0:
        rows += 1
    cfg = flat_cfg(din, dout)
    desc = describe(rows, cols, din, dout, cfg)
    assert desc.startswith("small") and "flat=1 " in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols * 7 + rows)
    y = R.softmax(x.to(DEV), out_dtype=DT[dout], config=cfg)
    torch.cuda.synchronize()
    assert_parity(x, y, dout, f"flat {rows}x{cols} {din}->{dout} [{desc}]")


def test_flat_widest_bf16_rows():
    # 1023 bf16 columns: 64 lanes of 16 elements in the row phase, one row a
    # tile
    rows, cols = 777, 1023
    cfg = flat_cfg("bf16", "bf16")
    desc = describe(rows, cols, "bf16", "bf16", cfg)
    assert "flat=1 " in desc and "lpr=64 " in desc and "nv=16 " in desc, desc
    x = W.random_matrix(rows, cols, "bf16", sigma=4.0, seed=cols)
    y = R.softmax(x.to(DEV), out_dtype=torch.bfloat16, config=cfg)
    torch.cuda.synchronize()
    assert_parity(x, y, "bf16", f"flat {rows}x{cols} [{desc}]")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("cols", [21, 77, 257])
def test_flat_log_softmax(cols, din, dout):
    rows = 1000 + 3
    cfg = flat_cfg(din, dout)
    desc = describe(rows, cols, din, dout, cfg, op=R.OP_LOG_SOFTMAX)
    assert "flat=1 " in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols)
    y = R.log_softmax(x.to(DEV), out_dtype=DT[dout], config=cfg)
    torch.cuda.synchronize()
    b = W.to_bits_numpy(x)
    xv = (oracle.widen_bf16_bits(b) if din == "bf16" else oracle.widen_f32(b)).reshape(rows, cols)
    v = oracle.log_softmax_f64(xv, threads=4)
    res = compare_log(widen_output(W.to_bits_numpy(y), dout).reshape(v.shape), v, dout)
    assert res["ok"], f"flat log {rows}x{cols} {din}->{dout} [{desc}]: {res}"


@pytest.mark.parametrize("din,dout", PAIRS)
def test_flat_special_values(din, dout):
    rows, cols = 64, 37
    x = W.random_matrix(rows, cols, "f32", sigma=3.0, seed=5)
    x[0, 5] = float("nan")
    x[1, 0] = float("inf")
    x[2, :] = float("-inf")
    x[3, ::3] = float("-inf")
    x[4, :] = 2.5
    x[5, :] = -1000.0
    x[5, cols // 2] = 0.0
    x[6, :-1] = float("-inf")
    x = x.to(DT[din])
    cfg = flat_cfg(din, dout)
    assert "flat=1 " in describe(rows, cols, din, dout, cfg)
    y = R.softmax(x.to(DEV), out_dtype=DT[dout], config=cfg)
    torch.cuda.synchronize()
    assert_parity(x, y, dout, f"flat special {din}->{dout}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_flat_in_place(dt):
    rows, cols = 4097, 77
    x = W.random_matrix(rows, cols, dt, sigma=5.0, seed=rows)
    xd = x.to(DEV)
    cfg = flat_cfg(dt, dt)
    assert "flat=1 " in describe(rows, cols, dt, dt, cfg)
    R.softmax(xd, out=xd, config=cfg)
    torch.cuda.synchronize()
    assert_parity(x, xd, dt, f"flat in place {rows}x{cols} {dt}")


@pytest.mark.parametrize("din,dout", PAIRS)
def test_flat_writes_only_the_output(din, dout):
    rows, cols = 999, 21
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=21)
    guard = 64
    buf = torch.full((guard + rows * cols + guard,), 7.0, dtype=DT[dout], device=DEV)
    out = buf[guard:guard + rows * cols].view(rows, cols)
    cfg = flat_cfg(din, dout)
    assert "flat=1 " in describe(rows, cols, din, dout, cfg)
    R.softmax(x.to(DEV), out=out, config=cfg)
    torch.cuda.synchronize()
    assert bool((buf[:guard] == 7.0).all()) and bool((buf[guard + rows * cols:] == 7.0).all())
    assert_parity(x, out, dout, f"flat guard {rows}x{cols} {din}->{dout}")


@pytest.mark.parametrize("din,dout", PAIRS)
def test_flat_by_configuration(din, dout):
    # the small variant at the full vector width asks for the flat form; a
    # grid cap given makes the blocks loop over tiles; narrow vectors asked
    # for keep the narrow plan; past 1024 columns the form is refused
    vw = full_vw(din, dout)
    rows, cols = 3001, 4 * vw + 1
    for cfg in (R.RowsmConfig(variant=R.SMALL, vw=vw),
                R.RowsmConfig(variant=R.SMALL, vw=vw, blocks_per_cu=1)):
        desc = describe(rows, cols, din, dout, cfg)
        assert "flat=1 " in desc, desc
        x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols)
        y = R.softmax(x.to(DEV), out_dtype=DT[dout], config=cfg)
        torch.cuda.synchronize()
        assert_parity(x, y, dout, f"flat forced {rows}x{cols} {din}->{dout} [{desc}]")
    assert "flat=0 " in describe(rows, cols, din, dout, R.RowsmConfig(vw=1))
    st, _ = R.rowsm_describe_op(R.OP_SOFTMAX, rows, 1025, R.dtype_code(DT[din]),
                                R.dtype_code(DT[dout]), R.RowsmConfig(variant=R.SMALL, vw=vw))
    assert st == R.EINVAL


@pytest.mark.parametrize("din,dout,cols", [("f32", "f32", 37), ("bf16", "bf16", 77),
                                           ("bf16", "f32", 9), ("f32", "bf16", 255),
                                           ("bf16", "bf16", 42)])
def test_flat_launcher_choice(din, dout, cols):
    # the launcher's own choice for 9-256 columns whose narrow vectors would
    # be of at most 4 bytes; sampled rows, the last ones among them, against
    # the oracle; every row's sum
    rows = 300007
    desc = describe(rows, cols, din, dout)
    assert desc.startswith("small") and "flat=1 " in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=3.0, seed=cols, device=DEV)
    y = R.softmax(x, out_dtype=DT[dout])
    torch.cuda.synchronize()
    sample = list(range(0, rows, 997)) + list(range(rows - 7, rows))
    assert_parity(x[sample].cpu(), y[sample].cpu(), dout, f"flat auto {rows}x{cols} [{desc}]")
    sums = y.double().sum(dim=1)
    tol = 1e-5 if dout == "f32" else 2.0 ** -8 * 2 + 1e-5
    assert float((sums - 1.0).abs().max()) <= tol


@pytest.mark.parametrize("slots", [2, 4])
@pytest.mark.parametrize("cols", [9, 21, 77, 255, 1017])
@pytest.mark.parametrize("op", [R.OP_SOFTMAX, R.OP_LOG_SOFTMAX])
def test_flat_bf16_tile_slots(op, cols, slots):
    # bf16 to bf16 tiles of 2 or 4 vectors per lane (rows_per_lane)
    g = (slots * 64 * 8 - 7) // cols
    rows = 3 * g + max(1, g // 2)
    if (rows * cols) % 8 == 0:
        rows += 1
    cfg = R.RowsmConfig(variant=R.SMALL, vw=8, rows_per_lane=slots)
    desc = describe(rows, cols, "bf16", "bf16", cfg, op=op)
    assert "flat=1 " in desc and f"rpl={slots} " in desc, desc
    x = W.random_matrix(rows, cols, "bf16", sigma=4.0, seed=cols + slots)
    if op == R.OP_SOFTMAX:
        y = R.softmax(x.to(DEV), config=cfg)
        torch.cuda.synchronize()
        assert_parity(x, y, "bf16", f"flat {rows}x{cols} slots {slots} [{desc}]")
    else:
        y = R.log_softmax(x.to(DEV), config=cfg)
        torch.cuda.synchronize()
        want = oracle.log_softmax_f64(oracle.widen_bf16_bits(W.to_bits_numpy(x)).reshape(rows, cols))
        res = compare_log(widen_output(W.to_bits_numpy(y), "bf16").reshape(rows, cols), want, "bf16")
        assert res["ok"], (desc, res)


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("cols", [9, 13, 15])
def test_flat_row_phase_lanes(cols, din, dout):
    # 9-16 columns: 4 lanes of 4 elements by default; 8 lanes of 2 asked for
    vw = full_vw(din, dout)
    if cols % vw == 0:
        pytest.skip("a multiple of the vector width")
    rows = 5000 + 3
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols + 1)
    for lanes, e in ((0, 4), (8, 2)):
        cfg = R.RowsmConfig(variant=R.SMALL, vw=vw, lanes_per_row=lanes)
        desc = describe(rows, cols, din, dout, cfg)
        assert f"lpr={lanes or 4} " in desc and f"nv={e} " in desc, desc
        y = R.softmax(x.to(DEV), out_dtype=DT[dout], config=cfg)
        torch.cuda.synchronize()
        assert_parity(x, y, dout, f"flat {rows}x{cols} {din}->{dout} [{desc}]")
