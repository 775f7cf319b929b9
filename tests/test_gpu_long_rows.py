"""GPU parity of the two-pass long-row form on rows of many tiles per thread:
2^22 columns with one 64-thread block per row and two vectors per tile (4096
to 8192 tiles per thread), and the launcher's own choice for such rows.  The
tolerances of log-softmax and the backward (oracle/compare.py) are derived for
every row length the ABI accepts; ascending rows make the running maximum
rise in every tile, and the nearly constant "creeping" rows make it rise by
about 1e-7 per tile: rescaling the running sum at each such rise lets the
rounding of the factor build up with the tile count."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_23089_amd as R
from oracle.compare import compare, compare_backward, compare_log, widen_output
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, PAIRS

pytestmark = pytest.mark.gpu

COLS = 1 << 22
ROWS = 2


def narrow_config():
    # one block of 64 threads per row, two vectors per tile: the most tiles
    # per thread a launch can have at this row length
    return R.RowsmConfig(variant=R.LARGE, split_blocks=-1, blocks_per_cu=1, block=64,
                         tile_vectors=2)


def rows_of(kind: str, din: str, seed: int) -> torch.Tensor:
    if kind == "random":
        return W.random_matrix(ROWS, COLS, din, sigma=4.0, seed=seed)
    if kind == "creeping":
        # nearly constant, rising by ~1e-7 from one tile of a thread to the
        # next: a sum rescaled at each rise would take a rescale factor just
        # below 1, rounded the same way, in every tile
        ramp = torch.linspace(0.0, 1e-3, COLS, dtype=torch.float64)
        x = torch.stack([ramp + 0.5 * r for r in range(ROWS)]).to(torch.float32)
        return x.to(DT[din])
    ramp = torch.linspace(-20.0, 20.0, COLS, dtype=torch.float64)
    if kind == "descending":
        ramp = ramp.flip(0)
    x = torch.stack([ramp + 3.0 * r for r in range(ROWS)]).to(torch.float32)
    return x.to(DT[din])


def widen_in(t: torch.Tensor) -> np.ndarray:
    b = W.to_bits_numpy(t)
    v = oracle.widen_bf16_bits(b) if t.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return v.reshape(-1, t.shape[-1])


def launch_desc(op, din, dout, cfg):
    st, desc = R.rowsm_describe_op(op, ROWS, COLS, R.dtype_code(DT[din]), R.dtype_code(DT[dout]),
                                   cfg)
    assert st == R.OK, desc
    return desc


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("kind", ["creeping", "ascending", "descending", "random"])
@pytest.mark.parametrize("shape", ["narrow", "auto"])
def test_softmax_and_log_many_tiles(shape, kind, din, dout):
    cfg = narrow_config() if shape == "narrow" else None
    desc = launch_desc(R.OP_LOG_SOFTMAX, din, dout, cfg)
    assert desc.startswith("large") and "split=0" in desc, desc
    if shape == "narrow":
        assert "block=64" in desc and "u=2" in desc and "stream=1" in desc, desc
    x = rows_of(kind, din, seed=17)
    xd = x.to(DEV)
    v_in = widen_in(x)
    y = R.log_softmax(xd, out_dtype=DT[dout], config=cfg)
    torch.cuda.synchronize()
    v = oracle.log_softmax_f64(v_in, threads=8)
    res = compare_log(widen_output(W.to_bits_numpy(y), dout).reshape(v.shape), v, dout)
    assert res["ok"], f"log {shape} {kind} {din}->{dout} [{desc}]: {res}"
    y = R.softmax(xd, out_dtype=DT[dout], config=cfg)
    torch.cuda.synchronize()
    v = oracle.softmax_f64(v_in, threads=8)
    res = compare(widen_output(W.to_bits_numpy(y), dout).reshape(v.shape), v, dout)
    assert res["ok"], f"softmax {shape} {kind} {din}->{dout} [{desc}]: {res}"
    # the sum of a row's probabilities, in fp64 over the fp32 output
    if dout == "f32":
        assert np.allclose(y.double().sum(dim=1).cpu().numpy(), 1.0, atol=1e-4)


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("shape", ["narrow", "auto"])
def test_backward_many_tiles(shape, din, dout):
    cfg = narrow_config() if shape == "narrow" else None
    desc = launch_desc(R.OP_SOFTMAX_BACKWARD, din, dout, cfg)
    assert desc.startswith("large") and "split=0" in desc, desc
    yp = W.random_probabilities(ROWS, COLS, din, 0.3, seed=5)
    dy = W.random_matrix(ROWS, COLS, din, sigma=1.0, seed=6)
    dx = R.softmax_backward(yp.to(DEV), dy.to(DEV), out_dtype=DT[dout], config=cfg)
    torch.cuda.synchronize()
    yw, dyw = widen_in(yp), widen_in(dy)
    v = oracle.softmax_backward_f64(yw, dyw, threads=8)
    res = compare_backward(widen_output(W.to_bits_numpy(dx), dout).reshape(v.shape), v, yw, dyw,
                           dout)
    assert res["ok"], f"backward {shape} {din}->{dout} [{desc}]: {res}"
