"""GPU parity of the flat short-row form of the softmax backward (rows of a
width that is not a multiple of the 16-byte vector width, y, dy and dx read
and written as streams of whole vectors aligned to the tensor and regrouped
into rows through LDS) against the fp64 oracle: every dtype pair, widths
from 1 to 1017-1023 columns with a partial final tile and a tensor that ends
inside a vector, in place over y and over dy, y and dy the same buffer,
special values, guard bands around dx, and the launcher's choice.
"""
import pytest
import torch

import paper_2607_23089_amd as R
from paper_2607_23089_amd import workloads as W
from test_gpu_backward import assert_bwd_parity, inputs, run_bwd
from test_gpu_parity import DEV, DT, PAIRS

pytestmark = pytest.mark.gpu


def full_vw(din, dout):
    return 16 // max(4 if din == "f32" else 2, 4 if dout == "f32" else 2)


def flat_cfg(din, dout):
    return R.RowsmConfig(variant=R.SMALL, vw=full_vw(din, dout))


def describe(rows, cols, din, dout, cfg=None):
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]), cfg)
    assert st == R.OK, desc
    return desc


def tile_rows(cols, vw):
    # three tiles and a partial fourth, the tensor ending inside a vector
    g = (4 * 64 * vw - (vw - 1)) // cols
    rows = 3 * g + max(1, g // 2)
    return rows + 1 if (rows * cols) % vw == 0 else rows


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("cols", [1, 3, 7, 9, 13, 21, 37, 41, 77, 129, 255, 257, 479, 513, 1017])
def test_bwd_flat_widths(cols, din, dout):
    vw = full_vw(din, dout)
    if cols % vw == 0:
        pytest.skip("a multiple of the vector width")
    rows = tile_rows(cols, vw)
    cfg = flat_cfg(din, dout)
    desc = describe(rows, cols, din, dout, cfg)
    assert desc.startswith("small") and "flat=1 " in desc, desc
    y, dy = inputs(rows, cols, din, seed=cols * 5 + rows)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout, config=cfg)
    assert_bwd_parity(y, dy, dx, dout, f"bwd flat {rows}x{cols} {din}->{dout} [{desc}]")


def test_bwd_flat_widest_bf16_rows():
    rows, cols = 555, 1023
    cfg = flat_cfg("bf16", "bf16")
    desc = describe(rows, cols, "bf16", "bf16", cfg)
    assert "flat=1 " in desc and "lpr=64 " in desc and "nv=16 " in desc, desc
    y, dy = inputs(rows, cols, "bf16", seed=3)
    dx = run_bwd(y.to(DEV), dy.to(DEV), "bf16", config=cfg)
    assert_bwd_parity(y, dy, dx, "bf16", f"bwd flat {rows}x{cols} [{desc}]")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("cols", [21, 77, 255])
def test_bwd_flat_in_place(cols, dt):
    rows = tile_rows(cols, full_vw(dt, dt))
    cfg = flat_cfg(dt, dt)
    y, dy = inputs(rows, cols, dt, seed=cols)
    yd, dyd = y.to(DEV), dy.to(DEV)
    run_bwd(yd, dyd, dt, config=cfg, out=dyd)
    assert_bwd_parity(y, dy, dyd, dt, f"bwd flat in place over dy {cols}")
    yd, dyd = y.to(DEV), dy.to(DEV)
    run_bwd(yd, dyd, dt, config=cfg, out=yd)
    assert_bwd_parity(y, dy, yd, dt, f"bwd flat in place over y {cols}")
    yd = y.to(DEV)
    dx = run_bwd(yd, yd, dt, config=cfg)
    assert_bwd_parity(y, y, dx, dt, f"bwd flat y == dy {cols}")


@pytest.mark.parametrize("din,dout", PAIRS)
def test_bwd_flat_special_values(din, dout):
    # a NaN in y makes its row NaN; an inf in dy makes d inf; nothing leaks
    # into the neighbouring rows of the tile
    rows, cols = 301, 37
    cfg = flat_cfg(din, dout)
    y, dy = inputs(rows, cols, din, seed=11)
    y[5, 3] = float("nan")
    dy[9, 0] = float("inf")
    dy[12, :] = 0.0
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout, config=cfg)
    assert_bwd_parity(y, dy, dx, dout, f"bwd flat special {din}->{dout}")
    dxc = dx.cpu().float()
    assert torch.isnan(dxc[5]).all()
    assert torch.all(dxc[12] == 0)
    assert torch.isfinite(dxc[4]).all() and torch.isfinite(dxc[6]).all()
    assert torch.isfinite(dxc[8]).all() and torch.isfinite(dxc[10]).all()


@pytest.mark.parametrize("cols", [13, 77])
def test_bwd_flat_bounded_writes(cols):
    rows = tile_rows(cols, 4) + 2
    y, dy = inputs(rows, cols, "f32", seed=cols)
    yd, dyd = y.to(DEV), dy.to(DEV)
    y0, dy0 = yd.clone(), dyd.clone()
    guard, n = 4096, rows * cols
    buf = torch.full((n + 2 * guard,), -123.0, device=DEV)
    dx = buf[guard:guard + n].view(rows, cols)
    run_bwd(yd, dyd, "f32", config=flat_cfg("f32", "f32"), out=dx)
    assert torch.all(buf[:guard] == -123.0) and torch.all(buf[guard + n:] == -123.0)
    assert torch.equal(yd, y0) and torch.equal(dyd, dy0)
    assert_bwd_parity(y, dy, dx, "f32", f"bwd flat bounded {cols}")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("rows,cols", [(204600, 41), (300001, 21), (20000, 77), (5000, 255),
                                       (3000, 479)])
def test_bwd_flat_launcher_choice(rows, cols, din, dout):
    desc = describe(rows, cols, din, dout)
    vw = full_vw(din, dout)
    # (bf16 to bf16: the flat form up to 128 columns, tiles of 2 vectors per
    # lane)
    bf = din == dout == "bf16"
    assert ("flat=1 " in desc) == (cols % vw != 0 and (not bf or cols <= 128)), desc
    if bf and "flat=1 " in desc:
        assert "rpl=2 " in desc, desc
    y, dy = inputs(rows, cols, din, seed=rows + cols)
    dx = run_bwd(y.to(DEV), dy.to(DEV), dout)
    assert_bwd_parity(y, dy, dx, dout, f"bwd launcher {rows}x{cols} {din}->{dout} [{desc}]")


def test_bwd_flat_misaligned_inputs_take_narrow_vectors():
    # y starting one element past a vector boundary: not the flat form
    rows, cols = 50, 37
    yb, dyb = inputs(1, rows * cols + 1, "f32", seed=2)
    y = yb.to(DEV).view(-1)[1:].view(rows, cols)
    dy = dyb.to(DEV).view(-1)[1:].view(rows, cols)
    dx = run_bwd(y, dy, "f32")
    assert_bwd_parity(y.cpu(), dy.cpu(), dx, "f32", "bwd misaligned odd width")
    with pytest.raises(R.RowsmError):
        run_bwd(y, dy, "f32", config=flat_cfg("f32", "f32"))


@pytest.mark.parametrize("slots", [2, 4])
@pytest.mark.parametrize("cols", [9, 41, 255, 1017])
def test_bwd_flat_bf16_tile_slots(cols, slots):
    # bf16 to bf16 tiles of 2 or 4 vectors per lane (rows_per_lane)
    g = (slots * 64 * 8 - 7) // cols
    rows = 3 * g + max(1, g // 2)
    if (rows * cols) % 8 == 0:
        rows += 1
    cfg = R.RowsmConfig(variant=R.SMALL, vw=8, rows_per_lane=slots)
    desc = describe(rows, cols, "bf16", "bf16", cfg)
    assert "flat=1 " in desc and f"rpl={slots} " in desc, desc
    y, dy = inputs(rows, cols, "bf16", seed=cols + slots)
    dx = run_bwd(y.to(DEV), dy.to(DEV), "bf16", config=cfg)
    assert_bwd_parity(y, dy, dx, "bf16", f"bwd flat {rows}x{cols} slots {slots} [{desc}]")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("cols", [9, 13])
def test_bwd_flat_row_phase_lanes(cols, din, dout):
    # 9-16 columns: 4 lanes of 4 elements by default; 8 lanes of 2 asked for
    vw = full_vw(din, dout)
    if cols % vw == 0:
        pytest.skip("a multiple of the vector width")
    rows = 4000 + 1
    y, dy = inputs(rows, cols, din, seed=cols + 2)
    for lanes, e in ((0, 4), (8, 2)):
        cfg = R.RowsmConfig(variant=R.SMALL, vw=vw, lanes_per_row=lanes)
        desc = describe(rows, cols, din, dout, cfg)
        assert f"lpr={lanes or 4} " in desc and f"nv={e} " in desc, desc
        dx = run_bwd(y.to(DEV), dy.to(DEV), dout, config=cfg)
        assert_bwd_parity(y, dy, dx, dout, f"bwd flat {rows}x{cols} [{desc}]")
