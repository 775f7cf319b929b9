"""GPU checks of rowsm_stream_copy, the measurement aid that the benchmark
times as each workload's copy ceiling: every dtype pair converts exactly
(bf16 -> f32 widening is exact, f32 -> bf16 rounds to nearest even, NaN stays
NaN), on vector and element paths, ragged lengths, misaligned views, in place,
and never writes past n."""
import numpy as np
import pytest
import torch

import paper_2607_23089_amd as R
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, PAIRS

pytestmark = pytest.mark.gpu


def expected_bits(x_cpu: torch.Tensor, dout: str) -> np.ndarray:
    """Bits of x converted to dout: widening by shifting the bf16 pattern,
    narrowing by round to nearest even on the fp32 pattern."""
    b = W.to_bits_numpy(x_cpu)
    if x_cpu.dtype == torch.bfloat16:
        f32 = b.astype(np.uint32) << 16
    else:
        f32 = b.view(np.uint32) if b.dtype != np.uint32 else b
    if dout == "f32":
        return f32.astype(np.uint32)
    r = ((f32.astype(np.uint64) + 0x7FFF + ((f32 >> 16) & 1)) >> 16).astype(np.uint16)
    return r


def got_bits(y: torch.Tensor) -> np.ndarray:
    b = W.to_bits_numpy(y.cpu())
    return b.view(np.uint32) if b.dtype == np.float32 else b


def special_values(n: int, dtype: str, seed: int) -> torch.Tensor:
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(n, generator=g) * 3.0
    sp = torch.tensor([float("inf"), -float("inf"), float("nan"), 0.0, -0.0, 1e-40, -1e-42,
                       3.4e38, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 2.0 ** -126])
    k = min(n, sp.numel())
    x[:k] = sp[:k]
    return x.to(DT[dtype])


def check(x_cpu, y_dev, dout, what):
    want = expected_bits(x_cpu, dout)
    got = got_bits(y_dev)
    fwant = want.astype(np.uint32) << (16 if dout == "bf16" else 0)
    fgot = got.astype(np.uint32) << (16 if dout == "bf16" else 0)
    nan_w = np.isnan(fwant.view(np.float32))
    nan_g = np.isnan(fgot.view(np.float32))
    assert np.array_equal(nan_w, nan_g), f"{what}: NaN positions differ"
    bad = (want != got) & ~nan_w
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {want.size} differ, first at "
                           f"{np.argwhere(bad)[:3].ravel().tolist()}")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("n", [1, 3, 255, 1024, 2047, 2048, 2049, 4099, (1 << 20) + 5])
@pytest.mark.parametrize("offset", [0, 1])
def test_stream_copy_exact(din, dout, n, offset):
    x = special_values(n + offset, din, seed=n)
    guard = 64
    y = torch.full((n + offset + guard,), 7.0, dtype=DT[dout], device=DEV)
    xd = x.to(DEV)
    st = R.rowsm_stream_copy(xd[offset:].data_ptr(), y[offset:].data_ptr(), n, R.dtype_code(x.dtype),
                             R.dtype_code(y.dtype), torch.cuda.current_stream().cuda_stream)
    assert st == R.OK
    torch.cuda.synchronize()
    check(x[offset:], y[offset:offset + n], dout, f"{din}->{dout} n={n} offset={offset}")
    tail = y[offset + n:].cpu().float()
    head = y[:offset].cpu().float()
    assert (tail == 7.0).all() and (head == 7.0).all(), "wrote outside [0, n)"


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_stream_copy_in_place_and_wrapper(dt):
    x = special_values(10000, dt, seed=5)
    xd = x.to(DEV)
    R.stream_copy(xd, out=xd)
    torch.cuda.synchronize()
    check(x, xd, dt, f"in place {dt}")
    for dout in ("f32", "bf16"):
        y = R.stream_copy(x.to(DEV).view(100, 100), out_dtype=DT[dout])
        torch.cuda.synchronize()
        assert y.shape == (100, 100) and y.dtype == DT[dout]
        check(x, y.view(-1), dout, f"wrapper {dt}->{dout}")
