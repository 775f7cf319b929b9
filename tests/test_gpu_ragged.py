"""GPU parity of the ragged-width form (rows whose width is not a multiple of
the 16-byte vector width, read in whole vectors aligned to the tensor with
element-wise row edges) against the fp64 oracle: every dtype pair, widths
leaving every remainder, row counts that put the row starts at every offset
inside a vector, softmax and log-softmax, in place, the form forced on rows
shorter than one vector, guard bands before and after the output, and the
launcher's own choice on a vocabulary-sized odd width.
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


def widen_in(t):
    b = W.to_bits_numpy(t)
    v = oracle.widen_bf16_bits(b) if t.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return v.reshape(-1, t.shape[-1])


def describe(rows, cols, din, dout, cfg=None, op=R.OP_SOFTMAX):
    st, desc = R.rowsm_describe_op(op, rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]),
                                   cfg)
    assert st == R.OK, desc
    return desc


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("extra", [1, 2, 3, 5, 7])
def test_ragged_widths_every_offset(extra, din, dout):
    # widths of a multiple of the vector width plus 1-7 elements (those that
    # are not multiples of it), spans of 300-2000 vectors; 2 vw + 3 rows put
    # the row starts at every offset inside a vector; every row against the
    # oracle
    vw = full_vw(din, dout)
    if extra % vw == 0:
        pytest.skip("a multiple of the vector width")
    for base in (300 * vw, 1000 * vw, 2000 * vw):
        cols = base + extra
        rows = 2 * vw + 3
        desc = describe(rows, cols, din, dout)
        assert "ragged=1 " in desc and f"vw={vw} " in desc, desc
        x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols + extra)
        y = R.softmax(x.to(DEV), out_dtype=DT[dout])
        torch.cuda.synchronize()
        assert_parity(x, y, dout, f"ragged {rows}x{cols} {din}->{dout} [{desc}]")


@pytest.mark.parametrize("din,dout", PAIRS)
def test_ragged_log_softmax(din, dout):
    vw = full_vw(din, dout)
    rows, cols = 3 * vw + 1, 700 * vw + vw - 1
    desc = describe(rows, cols, din, dout, op=R.OP_LOG_SOFTMAX)
    assert "ragged=1 " in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols)
    y = R.log_softmax(x.to(DEV), out_dtype=DT[dout])
    torch.cuda.synchronize()
    v = oracle.log_softmax_f64(widen_in(x), threads=4)
    res = compare_log(widen_output(W.to_bits_numpy(y), dout).reshape(v.shape), v, dout)
    assert res["ok"], f"ragged log {rows}x{cols} {din}->{dout} [{desc}]: {res}"


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_ragged_in_place(dt):
    vw = full_vw(dt, dt)
    rows, cols = 4 * vw + 3, 257 * vw + 1
    assert "ragged=1 " in describe(rows, cols, dt, dt)
    x = W.random_matrix(rows, cols, dt, sigma=4.0, seed=rows)
    xd = x.to(DEV)
    R.softmax(xd, out=xd)
    torch.cuda.synchronize()
    assert_parity(x, xd, dt, f"ragged in place {rows}x{cols} {dt}")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("cols", [1, 2, 3, 5, 13, 37, 131])
def test_ragged_forced_on_short_rows(cols, din, dout):
    # the form asked for by vector width on rows of fewer vectors than a wave
    # (one row spanning one or two vectors, both edges in one vector)
    vw = full_vw(din, dout)
    if cols % vw == 0:
        pytest.skip("a multiple of the vector width")
    cfg = R.RowsmConfig(vw=vw)
    rows = 4 * vw + 1
    desc = describe(rows, cols, din, dout, cfg)
    assert "ragged=1 " in desc and "medium" in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols + vw)
    y = R.softmax(x.to(DEV), out_dtype=DT[dout], config=cfg)
    torch.cuda.synchronize()
    assert_parity(x, y, dout, f"ragged forced {rows}x{cols} {din}->{dout} [{desc}]")


@pytest.mark.parametrize("din,dout", PAIRS)
def test_ragged_writes_only_the_output(din, dout):
    # output inside a larger buffer with guard bands of sentinel values before
    # and after it: the row edges are written element by element, nothing
    # outside the rows is touched, every row matches the oracle
    vw = full_vw(din, dout)
    rows, cols = 2 * vw + 1, 300 * vw + 3
    assert "ragged=1 " in describe(rows, cols, din, dout)
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=11)
    guard = 64  # elements: keeps the output 16-byte aligned
    buf = torch.full((guard + rows * cols + guard,), 7.0, dtype=DT[dout], device=DEV)
    out = buf[guard:guard + rows * cols].view(rows, cols)
    R.softmax(x.to(DEV), out=out)
    torch.cuda.synchronize()
    assert bool((buf[:guard] == 7.0).all()) and bool((buf[guard + rows * cols:] == 7.0).all())
    assert_parity(x, out, dout, f"ragged guard {rows}x{cols} {din}->{dout}")


def test_ragged_misaligned_views_keep_narrow_vectors():
    # a view one element past a 16-byte boundary cannot use the aligned
    # vector grid: the launcher keeps narrow vectors, and parity holds
    rows, cols = 9, 1203
    base = W.random_matrix(rows * cols + 1, 1, "bf16", sigma=4.0, seed=3).view(-1).to(DEV)
    x = base[1:].view(rows, cols)
    y = R.softmax(x)
    torch.cuda.synchronize()
    assert_parity(x.cpu(), y, "bf16", "misaligned ragged view")
    cfg = R.RowsmConfig(vw=8)
    with pytest.raises(R.RowsmError):
        R.softmax(x, config=cfg)


@pytest.mark.parametrize("din,dout,cols", [("bf16", "bf16", 40001), ("bf16", "f32", 32001),
                                           ("f32", "f32", 32001)])
def test_ragged_vocabulary_width(din, dout, cols):
    # odd vocabulary widths at a row count the launcher gives the ragged form:
    # sampled rows, the last ones among them, against the oracle; every row's
    # sum
    rows = 1031
    desc = describe(rows, cols, din, dout)
    assert "ragged=1 " in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=3.0, seed=7, device=DEV)
    y = R.softmax(x, out_dtype=DT[dout])
    torch.cuda.synchronize()
    sample = list(range(0, rows, 97)) + list(range(rows - 5, rows))
    assert_parity(x[sample].cpu(), y[sample].cpu(), dout, f"ragged vocab {rows}x{cols} [{desc}]")
    sums = y.double().sum(dim=1)
    tol = 1e-5 if dout == "f32" else 2.0 ** -8 * 4 + 1e-5
    assert float((sums - 1.0).abs().max()) <= tol


@pytest.mark.parametrize("din,dout,rows,cols", [("f32", "f32", 96, 30001),
                                                ("f32", "f32", 200, 38401),
                                                ("bf16", "f32", 200, 38401),
                                                ("bf16", "bf16", 64, 16385),
                                                ("f32", "bf16", 131, 24577)])
def test_ragged_few_long_rows(din, dout, rows, cols):
    # rows too long for one block's narrow vectors, from cus / 4 rows: the
    # ragged form on 8-16 waves (up to 10 slots of 4-element vectors), every
    # row against the oracle
    desc = describe(rows, cols, din, dout)
    assert desc.startswith("medium") and "ragged=1 " in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=rows + cols)
    y = R.softmax(x.to(DEV), out_dtype=DT[dout])
    torch.cuda.synchronize()
    assert_parity(x, y, dout, f"ragged few rows {rows}x{cols} {din}->{dout} [{desc}]")
