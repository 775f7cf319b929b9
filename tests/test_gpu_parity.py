"""GPU parity: every kernel family through the C ABI against the fp64 oracle.

Element-by-element comparison on seeded inputs that span several tiles and a
ragged tail, for every family the launcher can choose and every dtype pair,
plus the edge cases (empty, one column, odd widths and misaligned rows,
special values, in place).  Tolerances (oracle/compare.py): fp32 output
within 2e-6 absolute; bf16 output within one bf16 ulp of the oracle value;
NaN positions and exact zeros identical.
"""
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
PAIRS = [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"), ("f32", "bf16")]


def oracle_of(x_cpu: torch.Tensor) -> np.ndarray:
    b = W.to_bits_numpy(x_cpu)
    v = oracle.widen_bf16_bits(b) if x_cpu.dtype == torch.bfloat16 else oracle.widen_f32(b)
    return oracle.softmax_f64(v.reshape(-1, x_cpu.shape[-1]), threads=4)


def run(x_dev, dout, variant=R.AUTO, config=None, out=None):
    y = R.softmax(x_dev, out_dtype=DT[dout], out=out, variant=variant, config=config)
    torch.cuda.synchronize()
    return y


def assert_parity(x_cpu, y_dev, dout, what=""):
    v = oracle_of(x_cpu)
    y = widen_output(W.to_bits_numpy(y_dev), dout).reshape(v.shape)
    res = compare(y, v, dout)
    assert res["ok"], f"{what}: {res}"
    return res


def family_accepts(rows, cols, din, dout, fam):
    st, _ = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]), fam)
    return st == R.OK


GRID_COLS = {
    R.SMALL: [1, 2, 3, 7, 8, 9, 16, 31, 32, 33, 63, 64, 65, 127, 128, 255, 256],
    R.MEDIUM: [1, 7, 33, 64, 200, 1000, 1023, 1024, 4095, 4096, 4097, 8200, 16385,
               65536, 151936],
    R.LARGE: [1, 7, 1000, 4097, 65536, 65540, 100003, 262144],
}


def grid_cases():
    for fam, cols_list in GRID_COLS.items():
        for din, dout in PAIRS:
            for cols in cols_list:
                for rows in (1, 3, 67):
                    if rows * cols > 3_000_000:
                        continue
                    yield fam, din, dout, rows, cols


@pytest.mark.parametrize("fam,din,dout,rows,cols", list(grid_cases()))
def test_family_grid(fam, din, dout, rows, cols):
    if not family_accepts(rows, cols, din, dout, fam):
        pytest.skip("family does not take this shape (checked by test_family_limits)")
    x = W.random_matrix(rows, cols, din, sigma=6.0, seed=rows * 7919 + cols)
    y = run(x.to(DEV), dout, variant=fam)
    assert_parity(x, y, dout, f"{R.VARIANT_NAMES[fam]} {rows}x{cols} {din}->{dout}")


def test_family_limits():
    # SMALL takes rows of at most 32 vectors, MEDIUM at most the registers of
    # 16 waves; anything else is refused without a launch.
    x = torch.zeros(4, 4096, device=DEV)
    y = torch.empty_like(x)
    st = R.rowsm_forward_variant(x.data_ptr(), y.data_ptr(), 4, 4096, R.F32, R.F32, 0, R.SMALL)
    assert st == R.EINVAL
    x = torch.zeros(2, 70000, device=DEV)
    y = torch.empty_like(x)
    st = R.rowsm_forward_variant(x.data_ptr(), y.data_ptr(), 2, 70000, R.F32, R.F32, 0, R.MEDIUM)
    assert st == R.EINVAL


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("fam", [R.SMALL, R.MEDIUM, R.LARGE, "two_pass", "two_pass_1block"])
def test_special_values(fam, din, dout):
    cols = {R.SMALL: 48, R.MEDIUM: 1000}.get(fam, 70000)
    x = W.random_matrix(8, cols, "f32", sigma=3.0, seed=11)
    x[0, 5] = float("nan")
    x[1, 0] = float("inf")
    x[2, :] = float("-inf")
    x[3, ::3] = float("-inf")           # masked entries with a finite max
    x[4, :] = 2.5                       # constant row
    x[5, :] = -1000.0
    x[5, cols // 2] = 0.0               # dominant entry
    x[6, :-1] = float("-inf")           # single finite entry, at the end
    x = x.to(DT[din])
    if fam == "two_pass":
        y = run(x.to(DEV), dout, config=R.RowsmConfig(variant=R.LARGE, split_blocks=-1))
    elif fam == "two_pass_1block":
        y = run(x.to(DEV), dout, config=R.RowsmConfig(variant=R.LARGE, split_blocks=-1,
                                                      blocks_per_cu=1))
    else:
        y = run(x.to(DEV), dout, variant=fam)
    assert_parity(x, y, dout, f"special {fam} {din}->{dout}")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("fam,cols", [(R.SMALL, 64), (R.MEDIUM, 4096), (R.LARGE, 70000),
                                      ("two_pass", 70000)])
def test_subnormal_exponent_range(fam, cols, din, dout):
    # entries spread evenly over x - max in [-110, 0]: exp(x - max) passes
    # through the fp32 subnormal range (x - max in [-103.3, -87.3]) and
    # underflows to zero below it; the comparator accepts flush to zero only
    # where the fp64 value is itself below 2^-126
    rows = 6
    g = torch.Generator().manual_seed(cols)
    base = torch.linspace(-110.0, 0.0, cols).repeat(rows, 1)
    x = base[:, torch.randperm(cols, generator=g)] + torch.arange(rows).view(-1, 1) * 7.5
    x = x.to(DT[din])
    if fam == "two_pass":
        y = run(x.to(DEV), dout, config=R.RowsmConfig(variant=R.LARGE, split_blocks=-1))
    else:
        y = run(x.to(DEV), dout, variant=fam)
    res = assert_parity(x, y, dout, f"subnormal range {fam} {cols} {din}->{dout}")
    v = oracle_of(x)
    assert (v[(v > 0) & (v < 2.0 ** -126)]).size > 0     # the row does reach it


@pytest.mark.parametrize("din,dout", PAIRS)
def test_misaligned_rows_fall_back_to_narrow_vectors(din, dout):
    # A view starting one element into its storage breaks 8/16-byte alignment;
    # the launcher must pick single-element accesses and stay exact.
    for fam, cols in ((R.SMALL, 24), (R.MEDIUM, 1024), (R.LARGE, 65600)):
        base = W.random_matrix(1, 5 * cols + 1, din, sigma=2.0, seed=cols).to(DEV)
        x = base.view(-1)[1:].view(5, cols)
        assert x.data_ptr() % 8 != 0
        y = run(x, dout, variant=fam)
        assert_parity(x.cpu(), y, dout, f"misaligned {R.VARIANT_NAMES[fam]} {din}->{dout}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("fam,cols", [(R.SMALL, 64), (R.MEDIUM, 4096), (R.LARGE, 80000)])
def test_in_place(fam, cols, dt):
    x = W.random_matrix(9, cols, dt, sigma=5.0, seed=3)
    xd = x.to(DEV)
    run(xd, dt, variant=fam, out=xd)
    assert_parity(x, xd, dt, f"in place {R.VARIANT_NAMES[fam]}")


def test_empty_and_degenerate():
    for rows, cols in ((0, 16), (16, 0), (0, 0)):
        x = torch.empty(rows, cols, device=DEV)
        y = torch.full((rows, cols), 7.0, device=DEV)
        assert R.rowsm_forward(x.data_ptr(), y.data_ptr(), rows, cols, R.F32, R.F32, 0) == R.OK
    x = W.random_matrix(300, 1, "f32", sigma=50.0, seed=1)
    y = run(x.to(DEV), "f32")
    assert_parity(x, y, "f32", "one column")


@pytest.mark.parametrize("cfg", [
    dict(variant=R.SMALL, lanes_per_row=16, rows_per_lane=1),
    dict(variant=R.SMALL, lanes_per_row=32, rows_per_lane=8, blocks_per_cu=1),
    dict(variant=R.SMALL, rows_per_lane=2, blocks_per_cu=1),
    dict(variant=R.SMALL, block=64, rows_per_lane=1),
    dict(variant=R.SMALL, block=128, rows_per_lane=8, blocks_per_cu=1),
    dict(variant=R.MEDIUM, waves_per_row=1, rows_per_block=8, blocks_per_cu=1),
    dict(variant=R.MEDIUM, waves_per_row=2, blocks_per_cu=1),
    dict(variant=R.MEDIUM, waves_per_row=16),
    dict(variant=R.MEDIUM, waves_per_row=4, rows_per_block=3, blocks_per_cu=1),
    dict(variant=R.LARGE, split_blocks=-1, block=256, tile_vectors=8, blocks_per_cu=1),
    dict(variant=R.LARGE, split_blocks=-1, block=1024, tile_vectors=2),
    dict(variant=R.LARGE, split_blocks=-1, block=64, tile_vectors=4, blocks_per_cu=1),
    dict(variant=R.LARGE, split_blocks=1, block=1024),
    dict(variant=R.LARGE, split_blocks=2, block=1024),
    dict(variant=R.LARGE, split_blocks=7, block=128, blocks_per_cu=1),
    dict(variant=R.LARGE, split_blocks=64, block=64),
    dict(variant=R.LARGE, blocks_per_cu=1),
])
def test_launch_overrides(cfg):
    # Overrides change the launch shape, never the result; blocks_per_cu=1
    # makes every block loop over several rows or row groups.
    cols = {R.SMALL: 64, R.MEDIUM: 3000, R.LARGE: 20000}[cfg["variant"]]
    if cfg.get("split_blocks", 0) >= 1:
        cols = 40000
    for din, dout in (("bf16", "bf16"), ("f32", "f32")):
        rows = 2500 if cfg["variant"] != R.LARGE else 600
        x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols)
        y = run(x.to(DEV), dout, config=R.RowsmConfig(**cfg))
        assert_parity(x, y, dout, f"override {cfg} {din}->{dout}")


def test_deterministic_and_bounded_writes():
    # Same input twice -> bitwise-identical output; nothing written outside y;
    # x untouched.
    for fam, cols in ((R.SMALL, 64), (R.MEDIUM, 4096), (R.LARGE, 151936), (R.LARGE, 262144)):
        rows = max(2, 2_000_000 // cols)
        x = W.random_matrix(rows, cols, "bf16", sigma=8.0, seed=5).to(DEV)
        x_before = x.clone()
        guard = 4096
        n = rows * cols
        buf = torch.full((n + 2 * guard,), -123.0, device=DEV)
        y1 = buf[guard:guard + n].view(rows, cols)
        run(x, "f32", variant=fam, out=y1)
        y2 = run(x, "f32", variant=fam)
        assert torch.equal(y1, y2), R.VARIANT_NAMES[fam]
        assert torch.all(buf[:guard] == -123.0) and torch.all(buf[guard + n:] == -123.0)
        assert torch.equal(x, x_before)


@pytest.mark.parametrize("din,dout", PAIRS)
def test_two_pass_large_form(din, dout):
    # The streaming two-pass form is the fallback for rows too long for the
    # split form; check it on its own over widths with ragged tiles.
    # several blocks per row for few rows (8-16 at 9 x 70001 and 3 x 262144),
    # one block per row with a grid cap
    for cols in (5, 4097, 70001, 262144):
        rows = 3 if cols > 100000 else 9
        x = W.random_matrix(rows, cols, din, sigma=5.0, seed=cols + 1)
        for bpc in (0, 1):
            cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=-1, blocks_per_cu=bpc)
            st, desc = R.rowsm_describe_op(R.OP_SOFTMAX, rows, cols, R.dtype_code(DT[din]),
                                           R.dtype_code(DT[dout]), cfg)
            assert st == R.OK and "split=0" in desc
            stream = int(desc.split("stream=")[1].split()[0])
            assert stream == 1 if bpc else (stream >= 8 or cols <= 5000), desc
            y = run(x.to(DEV), dout, config=cfg)
            assert_parity(x, y, dout, f"two-pass {rows}x{cols} {din}->{dout} [{desc}]")


def test_split_many_launches_and_streams():
    # Consecutive split launches (new epoch each) on alternating streams reuse
    # the device workspace; each result must be exact, and repeated launches
    # on the same data bitwise equal.
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    xs = [W.random_matrix(37, 33000 + 8 * i, "bf16", sigma=4.0, seed=i).to(DEV)
          for i in range(4)]
    ys = []
    for it in range(12):
        s = s1 if it % 2 == 0 else s2
        x = xs[it % 4]
        with torch.cuda.stream(s):
            ys.append(R.softmax(x, out_dtype=torch.float32, variant=R.LARGE, stream=s))
    torch.cuda.synchronize()
    for it, y in enumerate(ys):
        if it < 4:
            assert_parity(xs[it].cpu(), y, "f32", f"split launch {it}")
        else:
            assert torch.equal(y, ys[it % 4])


def test_streams():
    # The kernel runs on the stream it is given.
    s = torch.cuda.Stream()
    x = W.random_matrix(512, 1000, "f32", seed=9).to(DEV)
    with torch.cuda.stream(s):
        y = R.softmax(x, stream=s)
    s.synchronize()
    assert_parity(x.cpu(), y, "f32", "side stream")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("rows,cols", [(1, 65536), (5, 65536), (40, 65536), (1, 151936),
                                       (17, 151936), (64, 151936), (3, 262144), (48, 262144)])
def test_few_rows_launcher_choice(rows, cols, din, dout):
    # few long rows: the launcher spreads each row over more blocks
    # (the row-count rules); parity in the launch it picks by itself
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
    assert st == R.OK
    x = W.random_matrix(rows, cols, din, sigma=5.0, seed=rows * 13 + cols)
    y = run(x.to(DEV), dout)
    assert_parity(x, y, dout, f"few rows {rows}x{cols} {din}->{dout} [{desc}]")


@pytest.mark.parametrize("din,dout", PAIRS)
@pytest.mark.parametrize("cols,S,bpc", [(65536, 8, 1), (151936, 8, 2), (262144, 32, 1),
                                        (100003, 16, 1), (40000, 2, 1)])
def test_split_prefetch_form(cols, S, bpc, din, dout):
    # the software-pipelined single-read form: each block loads its next row
    # during the current row's exchange; few blocks per compute unit so that
    # every block walks many rows
    rows = 300 if cols < 200000 else 120
    cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=S, blocks_per_cu=bpc, prefetch=1)
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]), cfg)
    if st != R.OK:
        pytest.skip("more values per lane than the prefetching form holds")
    assert "prefetch=1" in desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols + S)
    y = run(x.to(DEV), dout, config=cfg)
    assert_parity(x, y, dout, f"prefetch {rows}x{cols} S={S} {din}->{dout}")


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("rows", [63, 64, 65, 255, 256, 257])
@pytest.mark.parametrize("cols", [65536, 151936, 262144])
def test_row_count_boundaries(rows, cols, dt):
    # the row-count rules switch at cus / 4 and cus rows (256 compute units):
    # parity on every row at and around both thresholds, launcher's choice
    x = W.random_matrix(rows, cols, dt, sigma=3.0, seed=rows + cols)
    y = run(x.to(DEV), dt)
    assert_parity(x, y, dt, f"rows {rows} x {cols} {dt}")


@pytest.mark.parametrize("din,dout", [("f32", "f32"), ("bf16", "f32")])
@pytest.mark.parametrize("rows,cols,S", [(20000, 4096, 4), (300000, 256, 4)])
def test_split_grid_beyond_residency(rows, cols, S, din, dout):
    # The single-read form launches one group of S blocks per row: with
    # 64-thread blocks the grid holds far more blocks than the device does at
    # once (80000 groups' blocks), and past the workspace's 2^20 blocks the
    # groups loop over the rows (300000 rows x 4 blocks)
    cfg = R.RowsmConfig(variant=R.LARGE, split_blocks=S, block=64)
    st, desc = R.rowsm_describe_op(R.OP_SOFTMAX, rows, cols, R.dtype_code(DT[din]),
                                   R.dtype_code(DT[dout]), cfg)
    assert st == R.OK and f"split={S}" in desc and f"grid={min(rows, (1 << 20) // S) * S}" in desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=rows + S)
    y = run(x.to(DEV), dout, config=cfg)
    assert_parity(x, y, dout, f"split grid {rows}x{cols} S={S} {din}->{dout}")


@pytest.mark.parametrize("rows,din,dout", [(1, "f32", "f32"), (3, "bf16", "bf16"),
                                           (2, "bf16", "f32")])
def test_maximum_row_length(rows, din, dout):
    # cols = 2^30 - 1, the longest row the ABI accepts (offsets inside a row
    # are 32-bit byte offsets; a 4 GiB - 4 byte fp32 row); with several rows
    # the row bases lie past 4 GiB.  Closed form: zeros with one 1.0 per row
    # at a seeded column, so y = e^-1 / s at the zeros and 1 / s at the one,
    # s = (cols - 1) e^-1 + 1 (the rows' fp32 sums run over 2^30 terms).
    import math
    cols = (1 << 30) - 1
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("large"), desc
    assert R.rowsm_forward(0, 0, 1, 1 << 30, R.F32, R.F32, 0) == R.EINVAL  # one past the limit
    x = torch.zeros(rows, cols, dtype=DT[din], device=DEV)
    pos = [(r * 2654435761 + 12345) % cols for r in range(rows)]
    for r, p in enumerate(pos):
        x[r, p] = 1.0
    y = torch.empty(rows, cols, dtype=DT[dout], device=DEV)
    R.softmax(x, out=y)
    torch.cuda.synchronize()
    ssum = (cols - 1) * math.exp(-1.0) + 1.0
    v0, v1 = math.exp(-1.0) / ssum, 1.0 / ssum
    got, want = [], []
    for r, p in enumerate(pos):
        row = y[r]
        got.append(row[p].double().item())
        want.append(v1)
        for part in (row[:p], row[p + 1:]):
            if part.numel():
                got += [part.min().double().item(), part.max().double().item()]
                want += [v0, v0]
    del x, y
    torch.cuda.empty_cache()
    res = compare(np.array(got), np.array(want), dout)
    assert res["ok"], f"max row length {rows}x{cols} {din}->{dout} [{desc}]: {res} {got}"


@pytest.mark.parametrize("rows,din,dout,cols,want,fam", [
    (2, "f32", "f32", 1 << 21, "split=64", R.AUTO),     # 64 blocks x 512 x 64 values
    (2, "f32", "f32", (1 << 21) + 4, "split=0", R.AUTO),  # one vector more: two passes
    (2, "bf16", "bf16", 1 << 21, "split=64", R.AUTO),
    (2, "bf16", "f32", 64 * 512 * 40, "split=64", R.AUTO),  # widening: 40 values per lane
    (2, "bf16", "f32", 64 * 512 * 40 + 4, "split=0", R.AUTO),
    (65, "bf16", "bf16", 196608, "packed=1", R.MEDIUM),  # packed medium: 24 slots x 1024
    (65, "bf16", "bf16", 196616, "large", R.AUTO),
    (3, "f32", "f32", 65536, "wpr=16", R.MEDIUM),       # 16 waves x 64 values
])
def test_form_capacity_limits(rows, din, dout, cols, want, fam):
    # the largest rows each register-resident form holds, and one vector more
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]), fam)
    assert st == R.OK and want in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols)
    y = run(x.to(DEV), dout, variant=fam)
    assert_parity(x, y, dout, f"capacity {rows}x{cols} {din}->{dout} [{desc}]")


@pytest.mark.parametrize("rows,cols,din,dout", [
    (2048, 32768, "f32", "f32"), (64, 65536, "bf16", "bf16"), (100, 151936, "bf16", "bf16"),
    (512, 65536, "bf16", "f32"), (300, 65536, "f32", "bf16")])
def test_wide_rows_take_split_form(rows, cols, din, dout):
    # rows that would need all 16 waves of one block: the launcher's own
    # choice at these row counts is the split form (about 128 bytes per lane)
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("large") and "split=0" not in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=rows + cols)
    y = run(x.to(DEV), dout)
    assert_parity(x, y, dout, f"wide rows {rows}x{cols} {din}->{dout} [{desc}]")


# Full launches of medium-length rows: one case per kind of measured launch
# shape (medium groups with one or two rows per block, the single-read form
# with one or two blocks per row), at 8201 rows (32 rows per compute unit of
# 256, an odd count).
MEASURED_SHAPES = [
    (1024, "f32", "f32", ("medium", "wpr=2 ", "block=128 ")),
    (2048, "f32", "f32", ("medium", "wpr=4 ", "block=512 ")),
    (2560, "f32", "f32", ("medium", "wpr=4 ", "block=256 ")),
    (4096, "f32", "f32", ("medium", "wpr=8 ", "block=512 ")),
    (6144, "f32", "f32", ("large", "split=1 ", "block=512 ")),
    (7680, "f32", "f32", ("large", "split=1 ", "block=512 ")),
    (8192, "f32", "f32", ("large", "split=2 ", "block=256 ")),
    (14336, "f32", "f32", ("large", "split=2 ", "block=256 ")),
    (16384, "f32", "f32", ("large", "split=2 ", "block=512 ")),
    (2560, "bf16", "bf16", ("medium", "wpr=4 ", "block=256 ")),
    (15360, "bf16", "bf16", ("large", "split=1 ", "block=512 ")),
    (32768, "bf16", "bf16", ("large", "split=4 ", "block=256 ")),
    (20480, "bf16", "bf16", ("large", "split=2 ", "block=256 ")),
    (18432, "bf16", "bf16", ("large", "split=2 ", "block=256 ")),
    (28672, "bf16", "bf16", ("large", "split=2 ", "block=256 ")),
    (24576, "bf16", "f32", ("large", "split=2 ", "block=512 ")),
    (3072, "bf16", "f32", ("medium", "wpr=4 ", "block=512 ")),
    (6144, "bf16", "f32", ("medium", "wpr=8 ", "vpl=3 ")),
    (9728, "bf16", "f32", ("large", "split=1 ", "block=512 ")),
    (10240, "bf16", "f32", ("large", "split=2 ", "block=256 ")),
    (16384, "bf16", "f32", ("large", "split=2 ", "block=256 ")),
    (11264, "bf16", "f32", ("large", "split=2 ", "block=256 ")),
    (3584, "f32", "bf16", ("medium", "wpr=4 ", "block=512 ")),
    (6656, "f32", "bf16", ("medium", "wpr=8 ", "vpl=4 ")),
    (11264, "f32", "bf16", ("large", "split=1 ", "block=512 ")),
    (12288, "f32", "bf16", ("large", "split=2 ", "block=256 ")),
    # lane fill: a smaller wave group when the table's leaves its last slot
    # mostly empty (256-thread blocks)
    (544, "bf16", "f32", ("medium", "wpr=1 ", "nv=3 ", "block=256 ")),    # 136 vectors
    (1152, "f32", "bf16", ("medium", "wpr=2 ", "nv=3 ", "block=256 ")),   # 288 vectors
    (2176, "bf16", "bf16", ("medium", "wpr=2 ", "nv=3 ", "block=256 ")),  # 272 vectors
    (1120, "f32", "f32", ("medium", "wpr=2 ", "nv=3 ", "block=256 ")),    # 280 vectors
]


@pytest.mark.parametrize("cols,din,dout,want", MEASURED_SHAPES)
def test_measured_launch_shapes(cols, din, dout, want):
    rows = 8201
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
    assert st == R.OK and all(w in desc for w in want), desc
    print(f"measured shape {rows}x{cols} {din}->{dout}: {desc}", flush=True)
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=cols + rows, device=DEV)
    y = run(x, dout)
    sample = list(range(0, rows, 97)) + [rows - 2, rows - 1]
    assert_parity(x[sample].cpu(), y[sample].cpu(), dout, f"{rows}x{cols} {din}->{dout} [{desc}]")
    sums = y.double().sum(dim=1)
    tol = 1e-5 if dout == "f32" else 2.0 ** -8 + 1e-5
    assert float((sums - 1.0).abs().max()) <= tol
    del x, y


@pytest.mark.parametrize("rows,cols,din,dout,want", [
    (1024, 8192, "bf16", "bf16", ("wpr=4 ", "vpl=4 ")),
    (2048, 12288, "bf16", "bf16", ("wpr=2 ", "packed=1 ")),
    (1531, 4096, "f32", "f32", ("wpr=2 ", "vpl=8 ")),
    (3001, 14336, "bf16", "f32", ("wpr=4 ", "vpl=14 "))])
def test_few_rows_per_cu_shapes(rows, cols, din, dout, want):
    # launches of 4-16 rows per compute unit: few waves per row, many bytes
    # per lane (the packed bf16 form among them); every row against the oracle
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("medium") and all(w in desc for w in want), desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=rows + cols, device=DEV)
    y = run(x, dout)
    sample = list(range(0, rows, 7)) + [rows - 1]
    assert_parity(x[sample].cpu(), y[sample].cpu(), dout, f"{rows}x{cols} {din}->{dout} [{desc}]")


@pytest.mark.parametrize("rows,cols,din,dout,want", [
    (1000003, 74, "f32", "f32", ("block=512 ", "grid=18432 ")),
    (700001, 156, "bf16", "bf16", ("block=512 ", "grid=13312 ")),
    (500001, 148, "bf16", "f32", ("block=512 ", "grid=14336 ")),
    (600011, 102, "f32", "bf16", ("block=512 ", "grid=11264 ")),
    (500003, 144, "f32", "f32", ("block=512 ", "grid=17408 ")),
    (300007, 168, "f32", "f32", ("block=512 ", "grid=12288 ")),
    (500001, 256, "f32", "bf16", ("block=512 ", "grid=23552 ")),
    (400009, 256, "f32", "f32", ("block=512 ", "grid=24576 ")),
    (250001, 512, "bf16", "bf16", ("block=512 ", "grid=15360 ")),
    (400009, 302, "f32", "f32", ("block=512 ", "grid=30720 "))])      # three slots
def test_one_wave_short_rows(rows, cols, din, dout, want):
    # one wave per row and one to four slots: a grid of about 32 KiB of
    # traffic per block in whole residencies, whose waves loop over many
    # rows each (ragged row counts, rows of whole 128-byte lines and of parts
    # of lines); sampled rows, the last ones among them, against the oracle,
    # every row's sum
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("medium") and "wpr=1 " in desc, desc
    assert all(w in desc for w in want), desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=rows + cols, device=DEV)
    y = run(x, dout)
    sample = list(range(0, rows, 4999)) + list(range(rows - 7, rows))
    assert_parity(x[sample].cpu(), y[sample].cpu(), dout, f"{rows}x{cols} {din}->{dout} [{desc}]")
    sums = y.double().sum(dim=1)
    tol = 1e-5 if dout == "f32" else 2.0 ** -8 * 2 + 1e-5
    assert float((sums - 1.0).abs().max()) <= tol
    del x, y


@pytest.mark.parametrize("rows,cols,din,dout,grid", [
    (1048583, 20, "bf16", "bf16", 6144), (2000003, 14, "f32", "f32", 14336),
    (1500007, 26, "f32", "f32", 18432), (800011, 30, "f32", "bf16", 8192)])
def test_small_rows_of_part_lines(rows, cols, din, dout, grid):
    # small rows of narrow (8-byte) vectors whose stores cover parts of
    # 128-byte lines: a grid of about 16 KiB of traffic per block in whole
    # residencies of 8 blocks per compute unit, whose waves loop over many
    # row groups;
    # the output prefilled with NaN so that every row is seen written,
    # sampled rows (the last ones among them) against the oracle
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("small") and f"block=256 grid={grid} " in desc, desc
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=rows + cols, device=DEV)
    y = torch.full((rows, cols), float("nan"), dtype=DT[dout], device=DEV)
    run(x, dout, out=y)
    assert bool(torch.isfinite(y).all())
    sample = list(range(0, rows, 4999)) + list(range(rows - 7, rows))
    assert_parity(x[sample].cpu(), y[sample].cpu(), dout, f"{rows}x{cols} {din}->{dout} [{desc}]")
    del x, y


@pytest.mark.parametrize("rows,cols", [(4099, 64), (4099, 1000), (4099, 4097)])
def test_many_rows_grid_stride(rows, cols):
    # the small and medium families' default grid (a task per wave or block)
    # and a grid capped at one block per compute unit, whose waves stride
    # over more tasks than the grid covers
    x = W.random_matrix(rows, cols, "bf16", sigma=4.0, seed=rows + cols)
    for cfg in (None, R.RowsmConfig(blocks_per_cu=1)):
        y = run(x.to(DEV), "bf16", config=cfg)
        assert_parity(x, y, "bf16", f"{rows}x{cols} cfg={cfg is not None}")


def test_measured_single_read_picks_on_streams_and_threads():
    # the launcher's own single-read picks for full launches of medium-length
    # rows (one block of 512 threads, two of 256) from four host threads on
    # four streams, interleaved with medium launches: bitwise equal to the
    # same launches made one at a time
    import threading
    shapes = [(8192, 6144, "f32", "f32"), (8192, 20480, "bf16", "bf16"),
              (8192, 6144, "bf16", "bf16"), (9000, 4096, "f32", "f32")]
    xs, refs = [], []
    for rows, cols, din, dout in shapes:
        x = W.random_matrix(rows, cols, din, sigma=3.0, seed=rows + cols, device=DEV)
        xs.append(x)
        refs.append(run(x, dout))
    descs = [R.rowsm_describe(r, c, R.dtype_code(DT[i]), R.dtype_code(DT[o]))[1]
             for r, c, i, o in shapes]
    assert "split=1 " in descs[0] and "split=2 " in descs[1], descs
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for _ in range(5):
                    y = R.softmax(xs[i], out_dtype=DT[shapes[i][3]], stream=s)
                    s.synchronize()
                    if not torch.equal(y, refs[i]):
                        errors.append(f"thread {i} [{descs[i]}]: result differs")
                        return
        except Exception as e:  # noqa: BLE001 - reported below
            errors.append(f"thread {i}: {e!r}")

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a launching thread did not finish"
    assert not errors, errors
    for i, x in enumerate(xs):
        sample = [0, x.shape[0] // 2, x.shape[0] - 1]
        assert_parity(x[sample].cpu(), refs[i][sample].cpu(), shapes[i][3], f"shape {i}")


def test_split_launches_from_host_threads():
    # four host threads, each with its own stream, launch single-read split
    # softmax and backward concurrently (the C calls run without the GIL):
    # the per-device workspace lock, tag reservation and cross-stream
    # ordering must keep every result exact
    import threading
    shapes = [(9, 70000 + 16 * i) for i in range(4)]
    xs = [W.random_matrix(r, c, "f32", sigma=3.0, seed=c).to(DEV) for r, c in shapes]
    refs = [run(x, "f32", variant=R.LARGE) for x in xs]
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for _ in range(6):
                    y = R.softmax(xs[i], variant=R.LARGE, stream=s)
                    s.synchronize()
                    if not torch.equal(y, refs[i]):
                        errors.append(f"thread {i}: result differs")
                        return
        except Exception as e:  # noqa: BLE001 - reported below
            errors.append(f"thread {i}: {e!r}")

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    assert not any(t.is_alive() for t in threads), "a launching thread did not finish"
    assert not errors, errors
    for i, x in enumerate(xs):
        assert_parity(x.cpu(), refs[i], "f32", f"threaded shape {i}")


@pytest.mark.parametrize("rows,cols,din,dout,want", [
    (262144, 64, "bf16", "bf16", ("block=64 ", "rpl=1 ")),      # 64 MiB, one width
    (1048576, 64, "bf16", "bf16", ("block=64 ", "rpl=1 ")),     # 256 MiB
    (2097152, 16, "f32", "f32", ("block=64 ", "rpl=1 ")),       # 256 MiB
    (262144, 64, "bf16", "f32", ("block=128 ", "rpl=2 ")),      # 96 MiB, widening
    (109227, 64, "f32", "bf16", ("block=128 ", "rpl=2 ")),      # 40 MiB, narrowing
    (1398101, 32, "bf16", "f32", ("block=128 ", "rpl=2 ")),     # 256 MiB
    (65536, 64, "bf16", "f32", ("block=256 ", "rpl=4 ")),       # 24 MiB: default
])
def test_small_row_launch_picks(rows, cols, din, dout, want):
    # the launcher's small-row block and row-group picks by launch size and
    # dtype pair: sampled rows element by element, every row sums to one
    st, desc = R.rowsm_describe(rows, cols, R.dtype_code(DT[din]), R.dtype_code(DT[dout]))
    assert st == R.OK and desc.startswith("small") and all(w in desc for w in want), desc
    print(f"small pick {rows}x{cols} {din}->{dout}: {desc}", flush=True)
    x = W.random_matrix(rows, cols, din, sigma=4.0, seed=rows + cols, device=DEV)
    y = run(x, dout)
    sample = sorted({0, 1, 2, 3, 5, 7, rows // 3, rows // 2, rows - 3, rows - 2, rows - 1}
                    | set(range(0, rows, max(1, rows // 61))))
    idx = torch.tensor(sample, device=DEV)
    assert_parity(x.index_select(0, idx).cpu(), y.index_select(0, idx).cpu(), dout,
                  f"{rows}x{cols} {din}->{dout} [{desc}]")
    sums = y.double().sum(dim=1)
    tol = 1e-5 if dout == "f32" else 2.0 ** -8 * 2 + 1e-5
    assert float((sums - 1.0).abs().max()) <= tol
    del x, y
