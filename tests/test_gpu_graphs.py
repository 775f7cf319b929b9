"""Every entry point captured into a HIP graph (torch.cuda.graph) and
replayed several times, with new inputs written eagerly and the device
synchronised between replays; every replay is checked against the fp64
oracle with the operation's tolerance.  Long rows keep the single-read split
form under capture (a region of the device's workspace ring, cleared by a
kernel recorded before each launch): captured replays are bitwise equal to
eager launches of the same plan, also with eager split launches (which reuse
the ring) and other graphs' replays in between, and any number of captured
exchanging launches can be recorded.
"""
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


def eager_split_launch():
    # a single-read launch outside capture (the first one creates the ring)
    x = torch.zeros(2, 262144, device=DEV)
    R.softmax(x, variant=R.LARGE)
    torch.cuda.synchronize()


SPLIT_CASES = [  # (op, rows, cols, din, dout)
    ("softmax", 300, 65540, "f32", "f32"),
    ("softmax", 64, 151936, "bf16", "f32"),
    ("log_softmax", 24, 262144, "f32", "bf16"),
    ("backward", 64, 262144, "f32", "f32"),
    ("backward", 40, 151936, "bf16", "bf16"),
]


def split_case(op, rows, cols, din, dout, seed):
    """Buffers, a launch closure and a refill for one single-read case."""
    x = torch.empty(rows, cols, dtype=DT[din], device=DEV)
    dy = torch.empty_like(x)
    y = torch.empty(rows, cols, dtype=DT[dout], device=DEV)

    def run(out=y, stream=None):
        if op == "softmax":
            R.softmax(x, out=out, stream=stream)
        elif op == "log_softmax":
            R.log_softmax(x, out=out, stream=stream)
        else:
            R.softmax_backward(x, dy, out=out, stream=stream)

    def refill(i):
        if op == "backward":
            x.copy_(W.random_probabilities(rows, cols, din, 0.1, seed=seed + i).to(DEV))
            dy.copy_(W.random_matrix(rows, cols, din, seed=seed + 50 + i).to(DEV))
        else:
            x.copy_(W.random_matrix(rows, cols, din, sigma=4.0, seed=seed + i).to(DEV))

    return x, dy, y, run, refill


@pytest.mark.parametrize("op,rows,cols,din,dout", SPLIT_CASES)
def test_captured_split_form_matches_eager(op, rows, cols, din, dout):
    eager_split_launch()
    code = {"softmax": R.OP_SOFTMAX, "log_softmax": R.OP_LOG_SOFTMAX,
            "backward": R.OP_SOFTMAX_BACKWARD}[op]
    st, desc = R.rowsm_describe_op(code, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]))
    assert st == R.OK and "split=" in desc and "split=0" not in desc, desc
    x, dy, y, run, refill = split_case(op, rows, cols, din, dout, seed=rows + cols)
    refill(0)
    g = capture(run)
    side = torch.cuda.Stream()
    y_eager = torch.empty_like(y)
    for i in range(4):
        refill(i)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        with torch.cuda.stream(side):          # eager split launch, shared workspace
            run(out=y_eager, stream=side)
        side.synchronize()
        assert torch.equal(y.view(torch.int16 if dout == "bf16" else torch.int32),
                           y_eager.view(torch.int16 if dout == "bf16" else torch.int32)), \
            f"{op} {rows}x{cols} replay {i}: captured single-read launch differs from eager"
    # and the last replay against the oracle
    xw = widen(x.cpu())
    if op == "softmax":
        res = compare(out_np(y, dout), oracle.softmax_f64(xw, threads=4), dout)
    elif op == "log_softmax":
        res = compare_log(out_np(y, dout), oracle.log_softmax_f64(xw, threads=4), dout)
    else:
        dyw = widen(dy.cpu())
        res = compare_backward(out_np(y, dout), oracle.softmax_backward_f64(xw, dyw, threads=4),
                               xw, dyw, dout)
    assert res["ok"], f"{op} {rows}x{cols}: {res}"


def test_two_graphs_with_split_launches_alternate():
    eager_split_launch()
    a = split_case("softmax", 64, 151936, "bf16", "f32", seed=7)
    b = split_case("backward", 64, 262144, "f32", "f32", seed=9)
    ga, gb = None, None
    a[4](0)
    b[4](0)
    ga, gb = capture(a[3]), capture(b[3])
    for i in range(6):
        a[4](i)
        b[4](i)
        torch.cuda.synchronize()
        (ga if i % 2 == 0 else gb).replay()
        (gb if i % 2 == 0 else ga).replay()
        torch.cuda.synchronize()
        for x, dy, y, run, _ in (a, b):
            ref = torch.empty_like(y)
            run(out=ref)
            torch.cuda.synchronize()
            assert torch.equal(y, ref), f"alternating graphs, round {i}"


def test_forced_split_form_under_capture():
    eager_split_launch()
    x = torch.zeros(4, 262144, device=DEV)
    y = torch.empty_like(x)
    y2 = torch.empty_like(x)
    statuses = []
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sh = torch.cuda.current_stream().cuda_stream
        cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=8)
        statuses.append(R.rowsm_forward_config(x.data_ptr(), y.data_ptr(), 4, 262144,
                                               R.F32, R.F32, sh, cfg))
        statuses.append(R.rowsm_forward(x.data_ptr(), y2.data_ptr(), 4, 262144,
                                        R.F32, R.F32, sh))
    assert statuses == [R.OK, R.OK]
    for _ in range(3):
        g.replay()
        torch.cuda.synchronize()
        assert torch.allclose(y, torch.full_like(y, 1.0 / 262144))
        assert torch.allclose(y2, torch.full_like(y2, 1.0 / 262144))


@pytest.mark.parametrize("rows,cols,din,dout,cfg,want", [
    # the launcher's own single-read pick with one block per row (a full
    # launch of 1536-vector rows)
    (40000, 6144, "f32", "f32", None, "split=1 "),
    # forced: one block per row, and two
    (1000, 3000, "bf16", "f32", dict(variant=R.LARGE, split_blocks=1), "split=1 "),
    (9000, 20480, "bf16", "bf16", None, "split=2 "),
])
def test_single_read_one_block_per_row_under_capture(rows, cols, din, dout, cfg, want):
    # every single-read launch exchanges through the workspace, one block
    # per row included: under capture it takes a ring region like any other,
    # and replays (with eager single-read launches in between) match eager
    # launches bitwise
    config = R.RowsmConfig(**cfg) if cfg else None
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]), config)
    assert st == R.OK and want in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols, device=DEV)
    y = torch.empty(rows, cols, dtype=DT[dout], device=DEV)
    ref = R.softmax(x, out_dtype=DT[dout], config=config).clone()
    g = capture(lambda: R.softmax(x, out=y, config=config))
    for i in range(3):
        y.zero_()
        eager_split_launch()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), f"replay {i} [{desc}]"


def test_many_captured_exchanging_launches():
    # Captured exchanging launches take ring regions like eager ones and
    # nothing is reserved for a graph's lifetime: 80 graphs of one
    # 32768-block single-read launch each (80 MiB of exchange words, more
    # than the 64 MiB ring) all capture, and each replays exactly, with eager
    # launches reusing the ring in between.
    eager_split_launch()
    rows, cols = 4096, 4096
    x = W.random_matrix(rows, cols, "f32", sigma=4.0, seed=11, device=DEV)
    cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=8, block=64)
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX, rows, cols, R.F32, R.F32, cfg)
    assert st == R.OK and "grid=32768" in desc
    ref = R.softmax(x, config=cfg).clone()
    graphs, outs = [], []
    for k in range(80):
        y = torch.empty_like(x)
        status = []
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            status.append(R.rowsm_forward_config(x.data_ptr(), y.data_ptr(), rows, cols, R.F32,
                                                 R.F32, torch.cuda.current_stream().cuda_stream,
                                                 cfg))
        assert status[0] == R.OK, f"capture {k}"
        graphs.append(g)
        outs.append(y)
    for k in (0, 1, 40, 79, 0):
        outs[k].zero_()
        eager_split_launch()
        torch.cuda.synchronize()
        graphs[k].replay()
        torch.cuda.synchronize()
        assert torch.equal(outs[k], ref), f"graph {k}"
    res = compare(out_np(outs[79][::97].contiguous().cpu(), "f32"),
                  oracle.softmax_f64(widen(x[::97].contiguous().cpu()), threads=4), "f32")
    assert res["ok"], res
