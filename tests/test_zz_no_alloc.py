"""rowsm_forward_noalloc, the entry point for callers that cannot allocate,
through the C ABI: two calls in a row on the forms whose blocks exchange
partial results (the second with a smaller input) give exactly what
rowsm_forward gives for the same input, match the fp64 oracle, and leave the
device's free memory unchanged; the entry point also runs the other families,
in place, and under stream capture.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare, widen_output
from paper_2607_23089_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def free_bytes() -> int:
    hip = ctypes.CDLL("libamdhip64.so")
    free, total = ctypes.c_size_t(), ctypes.c_size_t()
    assert hip.hipMemGetInfo(ctypes.byref(free), ctypes.byref(total)) == 0
    return free.value


def call(fn, x, y):
    rows, cols = x.shape
    st = fn(x.data_ptr(), y.data_ptr(), rows, cols, R.dtype_code(x.dtype), R.dtype_code(y.dtype),
            torch.cuda.current_stream().cuda_stream)
    assert st == R.OK, R.rowsm_status_string(st)


def check_oracle(x, y, dout, step, what):
    xs = x[::step].contiguous().cpu()
    b = W.to_bits_numpy(xs)
    v = oracle.softmax_f64(oracle.widen_bf16_bits(b) if xs.dtype == torch.bfloat16
                           else oracle.widen_f32(b), threads=8)
    got = widen_output(W.to_bits_numpy(y[::step].contiguous().cpu()), dout).reshape(v.shape)
    res = compare(got, v, dout)
    assert res["ok"], f"{what}: {res}"


def test_two_calls_match_rowsm_forward():
    # exchanging forms: the vocabulary workload (32768 blocks, one row
    # group per row), then a smaller launch of 65540-wide rows
    shapes = [(4096, 151936, "bf16", "f32", 256), (64, 65540, "f32", "f32", 1)]
    inputs, outs, refs = [], [], []
    for rows, cols, din, dout, _ in shapes:
        st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
        assert st == R.OK and "split=" in desc and "split=0" not in desc, desc
        x = W.random_matrix(rows, cols, din, sigma=4.0, seed=rows + cols, device=DEV)
        inputs.append(x)
        outs.append(torch.full((rows, cols), float("nan"), dtype=DT[dout], device=DEV))
        refs.append(torch.empty(rows, cols, dtype=DT[dout], device=DEV))
    warm_x = W.random_matrix(8, 262144, "f32", seed=3, device=DEV)
    warm_y = torch.empty_like(warm_x)
    call(R.rowsm_forward_noalloc, warm_x, warm_y)     # set-up on this device
    for x, r in zip(inputs, refs):
        call(R.rowsm_forward, x, r)
    torch.cuda.synchronize()
    before = free_bytes()
    for x, y in zip(inputs, outs):                    # two calls in a row
        call(R.rowsm_forward_noalloc, x, y)
    torch.cuda.synchronize()
    assert free_bytes() == before, "rowsm_forward_noalloc changed the device's free memory"
    for (rows, cols, din, dout, step), x, y, r in zip(shapes, inputs, outs, refs):
        what = f"noalloc {rows}x{cols} {din}->{dout}"
        assert torch.equal(y.view(torch.int32), r.view(torch.int32)), f"{what} differs"
        check_oracle(x, y, dout, step, what)


@pytest.mark.parametrize("rows,cols,din,dout", [
    (262144, 64, "bf16", "bf16"), (64, 1000, "f32", "f32"), (512, 4096, "bf16", "bf16"),
    (24, 262144, "f32", "bf16"), (3, 1 << 22, "f32", "f32")])
def test_every_family(rows, cols, din, dout):
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols, device=DEV)
    y = torch.empty(rows, cols, dtype=DT[dout], device=DEV)
    r = torch.empty_like(y)
    call(R.rowsm_forward_noalloc, x, y)
    call(R.rowsm_forward, x, r)
    torch.cuda.synchronize()
    bits = torch.int16 if dout == "bf16" else torch.int32
    assert torch.equal(y.view(bits), r.view(bits))
    check_oracle(x, y, dout, max(1, rows // 64), f"noalloc {rows}x{cols}")


def test_in_place_and_errors():
    x = W.random_matrix(40, 151936, "f32", sigma=4.0, seed=5)
    xd = x.to(DEV)
    call(R.rowsm_forward_noalloc, xd, xd)
    torch.cuda.synchronize()
    check_oracle(x, xd, "f32", 1, "noalloc in place")
    assert R.rowsm_forward_noalloc(0, 0, 4, 4, R.F32, R.F32, 0) == R.EINVAL
    assert R.rowsm_forward_noalloc(0, 0, 0, 4, R.F32, R.F32, 0) == R.OK
    assert R.rowsm_forward_noalloc(1, 1, 4, 4, 7, R.F32, 0) == R.EDTYPE


def test_under_capture():
    srcs = [W.random_matrix(64, 151936, "bf16", sigma=3.0, seed=40 + i, device=DEV)
            for i in range(3)]
    x = srcs[0].clone()
    y = torch.empty(64, 151936, device=DEV)
    r = torch.empty_like(y)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(R.rowsm_forward_noalloc, x, y)
    for i in range(3):
        x.copy_(srcs[i])
        call(R.rowsm_forward, x, r)                   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, r), f"replay {i}"
