"""Every entry point captured into a HIP graph (torch.cuda.graph) and
replayed several times, with new inputs written eagerly and the device
synchronised between replays; every replay is checked against the fp64
oracle with the operation's tolerance.  Long rows take the two-pass form
under capture (the single-read form keeps per-launch host state); forcing the
single-read form there is refused."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare, compare_backward, compare_log, widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT

pytestmark = pytest.mark.gpu


def widen(t):
    b = W.to_bits_numpy(t)
    v = oracle.widen_bf16_bits(b) if t.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return v.reshape(-1, t.shape[-1])


def out_np(t, dt):
    return widen_output(W.to_bits_numpy(t), dt)


def capture(fn):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()                                   # eager warm-up before capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def replay_and_check(g, refill, check, replays=3):
    for i in range(replays):
        refill(i)                              # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        check(i)


FORWARD = [  # (name, rows, cols, din, dout)
    ("small", 4096, 64, "bf16", "bf16"),
    ("medium", 256, 4096, "bf16", "bf16"),
    ("large", 8, 262144, "f32", "f32"),
    ("vocab", 8, 151936, "bf16", "f32"),
]


@pytest.mark.parametrize("name,rows,cols,din,dout", FORWARD)
@pytest.mark.parametrize("op", ["softmax", "log_softmax", "scaled_causal"])
def test_forward_graph_replays(op, name, rows, cols, din, dout):
    x = torch.empty(rows, cols, dtype=DT[din], device=DEV)
    y = torch.empty(rows, cols, dtype=DT[dout], device=DEV)
    src = [W.random_matrix(rows, cols, din, sigma=4.0, seed=100 + i) for i in range(3)]
    x.copy_(src[0].to(DEV))
    period, offset = (rows, cols - rows) if op == "scaled_causal" else (0, 0)

    def run():
        if op == "softmax":
            R.softmax(x, out=y)
        elif op == "log_softmax":
            R.log_softmax(x, out=y)
        else:
            R.scaled_causal_softmax(x, 0.25, period, offset, out=y)

    g = capture(run)

    def check(i):
        v_in = widen(src[i])
        if op == "softmax":
            res = compare(out_np(y, dout), oracle.softmax_f64(v_in, threads=4), dout)
        elif op == "log_softmax":
            res = compare_log(out_np(y, dout), oracle.log_softmax_f64(v_in, threads=4), dout)
        else:
            v = oracle.softmax_scaled_causal_f64(v_in, 0.25, period, offset, threads=4)
            res = compare(out_np(y, dout), v, dout)
        assert res["ok"], f"{op} {name} replay {i}: {res}"

    replay_and_check(g, lambda i: x.copy_(src[i].to(DEV)), check)


@pytest.mark.parametrize("rows,cols,dt", [(4096, 64, "bf16"), (256, 4096, "bf16"),
                                          (8, 262144, "f32")])
def test_backward_graph_replays(rows, cols, dt):
    y = torch.empty(rows, cols, dtype=DT[dt], device=DEV)
    dy = torch.empty_like(y)
    dx = torch.empty_like(y)
    src = [(W.random_probabilities(rows, cols, dt, 0.1, seed=10 + i),
            W.random_matrix(rows, cols, dt, seed=20 + i)) for i in range(3)]

    def refill(i):
        y.copy_(src[i][0].to(DEV))
        dy.copy_(src[i][1].to(DEV))

    refill(0)
    g = capture(lambda: R.softmax_backward(y, dy, out=dx))

    def check(i):
        yw, dyw = widen(src[i][0]), widen(src[i][1])
        v = oracle.softmax_backward_f64(yw, dyw, threads=4)
        res = compare_backward(out_np(dx, dt), v, yw, dyw, dt)
        assert res["ok"], f"backward {rows}x{cols} replay {i}: {res}"

    replay_and_check(g, refill, check)


def test_moe_graph_replays():
    s = torch.empty(8192, 256, dtype=torch.bfloat16, device=DEV)
    o = torch.empty(8192, 8, dtype=torch.float32, device=DEV)
    src = [W.random_matrix(8192, 256, "bf16", seed=30 + i) for i in range(3)]
    s.copy_(src[0].to(DEV))
    g = capture(lambda: R.moe_group_top2(s, 32, out=o))

    def check(i):
        v = oracle.moe_group_top2_f64(widen(src[i]), 32, "f32")
        assert np.array_equal(o.cpu().double().numpy(), v), f"moe replay {i}"

    replay_and_check(g, lambda i: s.copy_(src[i].to(DEV)), check)


def test_forced_split_form_refused_under_capture():
    x = torch.zeros(4, 262144, device=DEV)
    y = torch.empty_like(x)
    statuses = []
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sh = torch.cuda.current_stream().cuda_stream
        cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=8)
        statuses.append(R.rowsm_forward_config(x.data_ptr(), y.data_ptr(), 4, 262144,
                                               R.F32, R.F32, sh, cfg))
        statuses.append(R.rowsm_forward(x.data_ptr(), y.data_ptr(), 4, 262144,
                                        R.F32, R.F32, sh))
    assert statuses == [R.EINVAL, R.OK]
    g.replay()
    torch.cuda.synchronize()
    assert torch.allclose(y, torch.full_like(y, 1.0 / 262144))
