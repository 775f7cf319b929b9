"""The exchanging LARGE forms (single-read split rows, and the two-pass form
with several blocks per row) when exchange waits give up, and their stream
contract.

With the wait limit set from the host to 0 (or a few polls), every wait (or
some of them) gives up and the block computes the missing partial results
from the input itself; the outputs must be bitwise equal to a launch whose
waits all succeeded, and match the fp64 oracle, for every form (softmax,
log-softmax, fused scale + causal mask, backward; one group per row, looping
groups, the prefetching form), and rowsm_split_wait_failures() must count the
give-ups.  In-place calls are never planned on an exchanging form: under a
zero wait limit they give up nothing.  Every kernel still exits normally: a
give-up only ends a wait.

The stream contract: the first exchanging call of a process returns while
another stream still runs a long kernel, without waiting for it; a first call
made under stream capture works (the exchange ring is a static device array:
nothing to allocate or clear first); launches on two streams with no ordering
between them give the right results.
"""
import json
import os
import subprocess
import sys
import textwrap

import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare, compare_backward, compare_log, widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def widen(t):
    b = W.to_bits_numpy(t)
    v = oracle.widen_bf16_bits(b) if t.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return v.reshape(-1, t.shape[-1])


def bits(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32)


class WaitLimit:
    """Sets the exchange wait limit for the duration of a with-block."""

    def __init__(self, polls):
        self.polls = polls

    def __enter__(self):
        torch.cuda.synchronize()
        self.prev = R.rowsm_set_split_wait_limit(self.polls)

    def __exit__(self, *exc):
        torch.cuda.synchronize()
        R.rowsm_set_split_wait_limit(self.prev)


# (name, op, rows, cols, din, dout, cfg): each plan exchanges between blocks
CASES = [
    ("split few rows", "softmax", 40, 151936, "bf16", "f32", None),
    ("split many rows", "softmax", 300, 65540, "f32", "f32", None),
    ("split looping groups", "softmax", 600, 65536, "f32", "bf16",
     dict(variant=R.LARGE, split_blocks=8, blocks_per_cu=1)),
    ("split prefetching", "softmax", 200, 131072, "bf16", "f32",
     dict(variant=R.LARGE, split_blocks=16, blocks_per_cu=1, prefetch=1)),
    ("split log", "log_softmax", 24, 262144, "f32", "bf16", None),
    ("split fused", "scaled_causal", 64, 151936, "bf16", "f32", None),
    ("two-pass blocks per row", "softmax", 4, 262144, "f32", "f32",
     dict(variant=R.LARGE, split_blocks=-1)),
    ("two-pass fused", "scaled_causal", 3, 262144, "bf16", "bf16",
     dict(variant=R.LARGE, split_blocks=-1)),
    ("two-pass log", "log_softmax", 2, 1 << 21, "f32", "f32", None),
    ("split backward", "backward", 64, 262144, "f32", "f32", None),
    ("split backward bf16", "backward", 40, 151936, "bf16", "bf16", None),
    ("two-pass backward", "backward", 4, 262144, "f32", "f32",
     dict(variant=R.LARGE, split_blocks=-1)),
]
OPS = {"softmax": R.OP_SOFTMAX, "log_softmax": R.OP_LOG_SOFTMAX,
       "scaled_causal": R.OP_SCALED_CAUSAL, "backward": R.OP_SOFTMAX_BACKWARD}


def exchanges(desc):
    return ("split=" in desc and "split=0" not in desc) or \
        ("stream=" in desc and "stream=0" not in desc and "stream=1 " not in desc)


def make_case(op, rows, cols, din, dout, seed):
    if op == "backward":
        y = W.random_probabilities(rows, cols, din, 0.1, seed=seed)
        dy = W.random_matrix(rows, cols, din, seed=seed + 1)
        return y, dy
    return W.random_matrix(rows, cols, din, sigma=4.0, seed=seed), None


def launch(op, x, dy, dout, cfg, out=None):
    config = R.RowsmConfig(**cfg) if cfg else None
    rows, cols = x.shape
    if op == "softmax":
        return R.softmax(x, out_dtype=DT[dout], out=out, config=config)
    if op == "log_softmax":
        return R.log_softmax(x, out_dtype=DT[dout], out=out, config=config)
    if op == "scaled_causal":
        return R.scaled_causal_softmax(x, 0.125, rows, cols - rows, out_dtype=DT[dout], out=out,
                                       config=config)
    return R.softmax_backward(x, dy, out_dtype=DT[dout], out=out, config=config)


def check_oracle(op, x, dy, y, dout, what):
    xw = widen(x)
    got = widen_output(W.to_bits_numpy(y.cpu()), dout).reshape(xw.shape)
    rows, cols = xw.shape
    if op == "softmax":
        res = compare(got, oracle.softmax_f64(xw, threads=8), dout)
    elif op == "log_softmax":
        res = compare_log(got, oracle.log_softmax_f64(xw, threads=8), dout)
    elif op == "scaled_causal":
        res = compare(got, oracle.softmax_scaled_causal_f64(xw, 0.125, rows, cols - rows,
                                                            threads=8), dout)
    else:
        dyw = widen(dy)
        res = compare_backward(got, oracle.softmax_backward_f64(xw, dyw, threads=8), xw, dyw,
                               dout)
    assert res["ok"], f"{what}: {res}"


@pytest.mark.forces_give_up
@pytest.mark.parametrize("name,op,rows,cols,din,dout,cfg", CASES, ids=[c[0] for c in CASES])
def test_given_up_waits_give_the_same_bits(name, op, rows, cols, din, dout, cfg):
    config = R.RowsmConfig(**cfg) if cfg else None
    st, desc = R.rowsm_describe_op(OPS[op], rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]), config)
    assert st == R.OK and exchanges(desc), f"{name}: {desc}"
    print(f"exchange give-up: {name} {rows}x{cols} {din}->{dout} [{desc}]", flush=True)
    x_cpu, dy_cpu = make_case(op, rows, cols, din, dout, seed=rows + cols)
    x = x_cpu.to(DEV)
    dy = dy_cpu.to(DEV) if dy_cpu is not None else None
    ref = launch(op, x, dy, dout, cfg)
    torch.cuda.synchronize()
    n0 = R.rowsm_split_wait_failures()
    for polls in (0, 1, 3):
        with WaitLimit(polls):
            y = launch(op, x, dy, dout, cfg)
        n1 = R.rowsm_split_wait_failures()
        assert torch.equal(bits(y), bits(ref)), f"{name}: limit {polls} changed the result"
        if polls == 0:
            assert n1 > n0, f"{name}: no wait gave up under a zero limit"
        n0 = n1
    check_oracle(op, x_cpu, dy_cpu, y, dout, name)


@pytest.mark.forces_give_up
@pytest.mark.parametrize("op,rows,cols,dt", [
    ("softmax", 40, 151936, "bf16"), ("softmax", 300, 65540, "f32"),
    ("log_softmax", 24, 262144, "f32"), ("scaled_causal", 64, 151936, "bf16"),
    ("backward", 64, 262144, "f32")])
def test_in_place_calls_do_not_exchange(op, rows, cols, dt):
    # Out of place, these shapes take an exchanging form; in place, the
    # launcher plans another one, so a zero wait limit gives nothing up.
    st, desc = R.rowsm_describe_op(OPS[op], rows, cols, R.dtype_code(DT[dt]),
                                   R.dtype_code(DT[dt]))
    assert st == R.OK and exchanges(desc), desc
    x_cpu, dy_cpu = make_case(op, rows, cols, dt, dt, seed=rows * 7 + cols)
    x = x_cpu.to(DEV)
    dy = dy_cpu.to(DEV) if dy_cpu is not None else None
    n0 = R.rowsm_split_wait_failures()
    with WaitLimit(0):
        if op == "backward":
            launch(op, x, dy, dt, None, out=dy)        # dx over dy
            y = dy
        else:
            launch(op, x, None, dt, None, out=x)
            y = x
    assert R.rowsm_split_wait_failures() == n0, f"in-place {op} took an exchanging form"
    check_oracle(op, x_cpu, dy_cpu, y, dt, f"in-place {op} {rows}x{cols}")
    if op == "softmax":
        # a forced single-read form in place is refused
        cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=4)
        st = R.rowsm_forward_config(x.data_ptr(), x.data_ptr(), rows, cols, R.dtype_code(DT[dt]),
                                    R.dtype_code(DT[dt]), 0, cfg)
        assert st == R.EINVAL


def test_two_streams_without_ordering():
    # launches on two streams, never ordered against each other, on the
    # exchanging forms: each output exact (the streams overlap in time)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    xa = W.random_matrix(64, 151936, "bf16", sigma=3.0, seed=1).to(DEV)
    xb = W.random_matrix(128, 262144, "f32", sigma=2.0, seed=2).to(DEV)
    ya_ref = R.softmax(xa, out_dtype=torch.float32)
    yb_ref = R.softmax(xb)
    torch.cuda.synchronize()
    outs = []
    for it in range(6):
        with torch.cuda.stream(s1):
            ya = R.softmax(xa, out_dtype=torch.float32, stream=s1)
        with torch.cuda.stream(s2):
            yb = R.softmax(xb, stream=s2)
        outs.append((ya, yb))
    torch.cuda.synchronize()
    for it, (ya, yb) in enumerate(outs):
        assert torch.equal(ya, ya_ref), f"stream 1 launch {it}"
        assert torch.equal(yb, yb_ref), f"stream 2 launch {it}"
    check_oracle("softmax", xa.cpu(), None, ya_ref, "f32", "two streams a")


CHILD_FIRST_CALL = textwrap.dedent("""
    import json, sys, time
    sys.path.insert(0, {root!r})
    import torch
    import paper_2607_23089_amd as R
    dev = torch.device("cuda:0")
    big = torch.ones(1 << 28, device=dev)          # 1 GiB
    dst = torch.empty_like(big)
    x = torch.randn(64, 151936, device=dev).to(torch.bfloat16)
    y = torch.empty(64, 151936, device=dev)
    torch.cuda.synchronize()
    busy, other = torch.cuda.Stream(), torch.cuda.Stream()
    with torch.cuda.stream(busy):
        for _ in range(60):                        # about 20 ms of copies
            R.check(R.rowsm_stream_copy(big.data_ptr(), dst.data_ptr(), big.numel(),
                                        R.F32, R.F32, busy.cuda_stream))
    t0 = time.perf_counter()
    st = R.rowsm_forward(x.data_ptr(), y.data_ptr(), 64, 151936, R.BF16, R.F32,
                         other.cuda_stream)
    dt_call = time.perf_counter() - t0
    busy_after_call = not busy.query()
    torch.cuda.synchronize()
    ref = torch.softmax(x.float(), dim=-1)
    err = (y - ref).abs().max().item()
    print(json.dumps(dict(status=st, call_ms=dt_call * 1e3, busy_after_call=busy_after_call,
                          max_err=err)))
""")

CHILD_FIRST_CAPTURE = textwrap.dedent("""
    import json, sys
    sys.path.insert(0, {root!r})
    import torch
    import paper_2607_23089_amd as R
    dev = torch.device("cuda:0")
    xs = [torch.randn(64, 151936, device=dev).to(torch.bfloat16) for _ in range(3)]
    x = torch.empty_like(xs[0])
    y = torch.empty(64, 151936, device=dev)
    x.copy_(xs[0])
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    status = []
    with torch.cuda.graph(g):                      # the process's first exchanging call
        status.append(R.rowsm_forward(x.data_ptr(), y.data_ptr(), 64, 151936, R.BF16, R.F32,
                                      torch.cuda.current_stream().cuda_stream))
    errs = []
    for i in range(3):
        x.copy_(xs[i])
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        errs.append((y - torch.softmax(xs[i].float(), dim=-1)).abs().max().item())
    print(json.dumps(dict(status=status[0], errs=errs,
                          failures=R.rowsm_split_wait_failures())))
""")


def run_child(src):
    res = subprocess.run([sys.executable, "-c", src.format(root=ROOT)], capture_output=True,
                         text=True, timeout=240)
    assert res.returncode == 0, res.stderr[-2000:]
    return json.loads(res.stdout.strip().splitlines()[-1])


def test_first_call_does_not_wait_for_other_streams():
    out = run_child(CHILD_FIRST_CALL)
    print(f"first exchanging call: {out}", flush=True)
    assert out["status"] == R.OK
    assert out["busy_after_call"], f"the first call waited for another stream: {out}"
    assert out["max_err"] <= 2e-6, out


def test_first_call_under_capture():
    out = run_child(CHILD_FIRST_CAPTURE)
    print(f"first exchanging call under capture: {out}", flush=True)
    assert out["status"] == R.OK and out["failures"] == 0
    assert max(out["errs"]) <= 2e-6, out
