"""GPU parity on seeded random shapes: every operation (softmax, log-softmax,
the fused scale + causal mask form, the backward) through the launcher's own
choice, at row counts and lengths drawn log-uniformly over the ranges its
rules split (1-40000 rows, 1-70000 columns, up to 120M elements), every dtype
pair, some views misaligned by one element.  Sampled rows are compared with
the fp64 oracle at each operation's tolerance; the launch each case takes is
printed first.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare, compare_backward, compare_log, widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, PAIRS

pytestmark = pytest.mark.gpu

OPS = ["softmax", "log_softmax", "scaled_causal", "backward"]
OP_CODE = {"softmax": R.OP_SOFTMAX, "log_softmax": R.OP_LOG_SOFTMAX,
           "scaled_causal": R.OP_SCALED_CAUSAL, "backward": R.OP_SOFTMAX_BACKWARD}


def draw_cases(n=96, seed=20261202):
    g = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        rows = int(np.exp(g.uniform(0.0, np.log(40000))))
        cols = int(np.exp(g.uniform(0.0, np.log(70000))))
        if rows * cols > 120_000_000:
            continue
        op = OPS[len(cases) % len(OPS)]
        din, dout = PAIRS[int(g.integers(len(PAIRS)))]
        misaligned = bool(g.random() < 0.2)
        cases.append((len(cases), op, rows, cols, din, dout, misaligned))
    return cases


def widen(t):
    b = W.to_bits_numpy(t)
    v = oracle.widen_bf16_bits(b) if t.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return v.reshape(-1, t.shape[-1])


def operand(rows, cols, dt, misaligned, make):
    """A rows x cols tensor from make(rows, cols), as a view one element into
    a larger buffer when misaligned."""
    if not misaligned:
        return make(rows, cols)
    buf = torch.empty(rows * cols + 1, dtype=DT[dt], device=DEV)
    v = buf[1:].view(rows, cols)
    v.copy_(make(rows, cols))
    return v


@pytest.mark.parametrize("case", draw_cases(), ids=lambda c: f"{c[0]}-{c[1]}-{c[2]}x{c[3]}")
def test_random_shape(case):
    _, op, rows, cols, din, dout, misaligned = case
    scale, period = 0.125, max(1, min(rows, cols))
    if op == "backward":
        y_in = operand(rows, cols, din, misaligned, lambda r, c: W.random_probabilities(
            r, c, din, 0.3, seed=rows + cols, device=DEV))
        dy = W.random_matrix(rows, cols, din, sigma=1.0, seed=rows + 2 * cols, device=DEV)
        ptrs = (y_in.data_ptr(), dy.data_ptr())
    else:
        x = operand(rows, cols, din, misaligned, lambda r, c: W.random_matrix(
            r, c, din, sigma=4.0, seed=rows + cols, device=DEV))
        ptrs = (x.data_ptr(),)
    out = torch.empty(rows * cols + (1 if misaligned else 0), dtype=DT[dout], device=DEV)
    y = out[1:].view(rows, cols) if misaligned else out.view(rows, cols)
    # the launch the library makes for these pointers
    st, desc = R.rowsm_describe_op(OP_CODE[op], rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    print(f"case {case}: plan for aligned pointers {desc if st == R.OK else st}", flush=True)
    sh = torch.cuda.current_stream().cuda_stream
    di, do = R.dtype_code(DT[din]), R.dtype_code(DT[dout])
    if op == "softmax":
        st = R.rowsm_forward(ptrs[0], y.data_ptr(), rows, cols, di, do, sh)
    elif op == "log_softmax":
        st = R.rowsm_log_softmax(ptrs[0], y.data_ptr(), rows, cols, di, do, sh)
    elif op == "scaled_causal":
        st = R.rowsm_forward_scaled_causal(ptrs[0], y.data_ptr(), rows, cols, di, do, scale,
                                           period, 0, sh)
    else:
        st = R.rowsm_softmax_backward(ptrs[0], ptrs[1], y.data_ptr(), rows, cols, di, do, sh)
    assert st == R.OK, R.rowsm_status_string(st)
    torch.cuda.synchronize()

    starts = sorted({0, rows // 3, rows // 2, max(0, rows - 3)})
    for r0 in starts:
        r1 = min(rows, r0 + 3)
        got = widen_output(W.to_bits_numpy(y[r0:r1].cpu()), dout).reshape(r1 - r0, cols)
        what = f"{op} {rows}x{cols} {din}->{dout} misaligned={misaligned} rows {r0}-{r1} [{desc}]"
        if op == "backward":
            yv, dyv = widen(y_in[r0:r1].cpu()), widen(dy[r0:r1].cpu())
            res = compare_backward(got, oracle.softmax_backward_f64(yv, dyv, threads=4), yv, dyv,
                                   dout)
        elif op == "log_softmax":
            res = compare_log(got, oracle.log_softmax_f64(widen(x[r0:r1].cpu()), threads=4), dout)
        elif op == "scaled_causal":
            v = oracle.softmax_scaled_causal_f64(widen(x[r0:r1].cpu()), scale, period, 0,
                                                 threads=4, row0=r0)
            res = compare(got, v, dout)
        else:
            res = compare(got, oracle.softmax_f64(widen(x[r0:r1].cpu()), threads=4), dout)
        assert res["ok"], f"{what}: {res}"
