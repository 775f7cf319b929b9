"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (rowsm_forward, the launcher's own choice).

Sampled rows are compared element by element with the fp64 oracle; every row
is checked for properties that hold at any size: no NaN, rows sum to one,
masked entries exactly zero (causal), the closed form 1/k at the k row
maxima and exactly 0 elsewhere (vocab outliers), the spike entry near one
(large rows).
"""
import numpy as np
import pytest
import torch

import paper_2607_23089_amd as R
from paper_2607_23089_amd import workloads as W
from test_gpu_parity import DEV, DT, assert_parity

pytestmark = pytest.mark.gpu


def sample_rows(w, n_random=8):
    g = np.random.default_rng(1234)
    rows = {0, 1, w.rows // 2, w.rows - 1}
    rows |= set(int(r) for r in g.integers(0, w.rows, n_random))
    if w.structure == "causal":
        rows |= {w.period - 1, w.period, 2 * w.period + 17}
    return sorted(r for r in rows if r < w.rows)


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_workload_full_size(name):
    w = W.WORKLOADS[name]
    print(f"workload {name}: {w.rows}x{w.cols} {w.in_dtype}->{w.out_dtype}", flush=True)
    x = W.make_input(w, device=DEV)
    y = torch.empty(w.rows, w.cols, dtype=DT[w.out_dtype], device=DEV)
    st = R.rowsm_forward(x.data_ptr(), y.data_ptr(), w.rows, w.cols,
                         R.dtype_code(x.dtype), R.dtype_code(y.dtype),
                         torch.cuda.current_stream().cuda_stream)
    assert st == R.OK
    torch.cuda.synchronize()

    rows = sample_rows(w)
    assert_parity(x[rows].cpu(), y[rows].cpu(), w.out_dtype, f"{name} rows {rows}")

    assert not torch.isnan(y).any()
    sums = y.double().sum(dim=1)
    tol = 1e-5 if w.out_dtype == "f32" else 2.0 ** -8 + 1e-5
    assert float((sums - 1.0).abs().max()) <= tol
    if w.structure == "causal":
        for r0 in range(0, w.rows, 4096):
            blk = y[r0:r0 + 4096]
            col = torch.arange(w.cols, device=DEV)
            lim = torch.arange(r0, r0 + blk.shape[0], device=DEV) % w.period
            masked = col[None, :] > lim[:, None]
            assert torch.all(blk[masked] == 0)
            del masked
    if w.structure == "outliers":
        for r0 in range(0, w.rows, 512):
            xb = x[r0:r0 + 512].float()
            yb = y[r0:r0 + 512]
            mx = xb.max(dim=1, keepdim=True).values
            assert torch.all(mx == 9984.0)
            at_max = xb == mx
            k = at_max.sum(dim=1, keepdim=True).double()
            want = (1.0 / k).expand_as(yb)
            assert float((yb.double() - want)[at_max].abs().max()) <= 2e-6
            assert torch.all(yb[~at_max] == 0)
    if w.structure == "spike":
        assert torch.all(y.max(dim=1).values >= 1.0 - 1e-6)
    del x, y
    torch.cuda.empty_cache()
