"""C ABI on the host (no GPU): the library loads, exports every declared
symbol, validates arguments before any HIP call, and the launcher's family
choice follows its stated thresholds."""
import ctypes
import os
import re

import pytest

import paper_2607_23089_amd as R

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "include", "rowsm.h")
MiB = 1 << 20


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(R.LIB_PATH):
        from paper_2607_23089_amd.build import build_library
        build_library()
    return R.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rowsm_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert set(names) == set(R.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_config_struct_matches_header():
    text = open(HEADER).read()
    body = re.search(r"typedef struct rowsm_config \{(.*?)\} rowsm_config;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"int32_t\s+(\w+);", body)
    assert fields == [f for f, _ in R.RowsmConfig._fields_]


def test_status_strings(lib):
    assert R.rowsm_status_string(R.OK) == "ok"
    assert "invalid" in R.rowsm_status_string(R.EINVAL)
    assert "dtype" in R.rowsm_status_string(R.EDTYPE)
    assert "HIP" in R.rowsm_status_string(R.EHIP)
    assert R.rowsm_status_string(12345) == "unknown status"


# Fake, never-dereferenced addresses: every call below must be rejected (or be
# a no-op) before the library makes any HIP call.  A case that would pass
# validation must never be added here: it would launch on these addresses.
X, Y = 0x7f0000000000, 0x7f8000000000


@pytest.mark.parametrize("args,want", [
    ((X, Y, 4, 8, 7, R.F32), R.EDTYPE),
    ((X, Y, 4, 8, R.F32, -1), R.EDTYPE),
    ((X, Y, -1, 8, R.F32, R.F32), R.EINVAL),
    ((X, Y, 4, -8, R.F32, R.F32), R.EINVAL),
    ((0, Y, 4, 8, R.F32, R.F32), R.EINVAL),
    ((X, 0, 4, 8, R.F32, R.F32), R.EINVAL),
    ((X, X + 4, 4, 8, R.F32, R.F32), R.EINVAL),          # partial overlap
    ((X, X, 4, 8, R.BF16, R.F32), R.EINVAL),             # in place, dtype change
    ((X, Y, 1, 1 << 30, R.F32, R.F32), R.EINVAL),        # row too long
    ((X, Y, 1 << 40, 1 << 23, R.F32, R.F32), R.EINVAL),  # rows*cols >= 2^62
    ((0, 0, 0, 8, R.F32, R.F32), R.OK),                  # empty: no launch
    ((0, 0, 8, 0, R.BF16, R.BF16), R.OK),
])
def test_argument_errors(lib, args, want):
    assert R.rowsm_forward(*args, 0) == want
    assert R.rowsm_forward_variant(*args, 0, R.AUTO) == want


def test_bad_variant_and_config(lib):
    assert R.rowsm_forward_variant(X, Y, 4, 8, R.F32, R.F32, 0, 9) == R.EINVAL
    assert R.rowsm_forward_variant(X, Y, 4, 8, R.F32, R.F32, 0, -2) == R.EINVAL
    # a family that cannot take the shape
    assert R.rowsm_forward_variant(X, Y, 4, 4096, R.F32, R.F32, 0, R.SMALL) == R.EINVAL
    assert R.rowsm_forward_variant(X, Y, 4, 1 << 20, R.F32, R.F32, 0, R.MEDIUM) == R.EINVAL
    bad = [dict(variant=R.SMALL, lanes_per_row=3), dict(variant=R.SMALL, lanes_per_row=64),
           dict(variant=R.SMALL, rows_per_lane=3), dict(variant=R.MEDIUM, waves_per_row=3),
           dict(variant=R.MEDIUM, waves_per_row=4, rows_per_block=8),
           dict(variant=R.LARGE, block=100), dict(variant=R.LARGE, tile_vectors=3),
           dict(variant=R.LARGE, block=2048), dict(variant=R.SMALL, rows_per_block=17),
           dict(variant=R.SMALL, block=512),
           dict(variant=R.LARGE, split_blocks=-2), dict(variant=R.MEDIUM, packed=2),
           dict(variant=R.SMALL, blocks_per_cu=-1), dict(variant=7),
           dict(variant=R.AUTO, vw=3), dict(variant=R.AUTO, vw=2),
           dict(variant=R.LARGE, split_blocks=65),
           dict(variant=R.MEDIUM, packed=1, waves_per_row=16)]
    for cfg in bad:
        st = R.rowsm_forward_config(X, Y, 64, 64, R.BF16, R.BF16, 0, R.RowsmConfig(**cfg))
        assert st == R.EINVAL, cfg


def test_scaled_causal_argument_errors(lib):
    f = R.rowsm_forward_scaled_causal
    assert f(X, Y, 4, 8, R.F32, R.F32, 0.5, -1, 0, 0) == R.EINVAL       # negative period
    assert f(X, Y, 4, 8, 9, R.F32, 0.5, 4, 0, 0) == R.EDTYPE
    assert f(X, Y, -4, 8, R.F32, R.F32, 0.5, 4, 0, 0) == R.EINVAL
    assert f(0, 0, 0, 8, R.F32, R.F32, 0.5, 4, 0, 0) == R.OK             # empty
    assert f(X, X + 4, 4, 8, R.F32, R.F32, 0.5, 4, 0, 0) == R.EINVAL     # overlap
    for cfg in (dict(variant=R.MEDIUM, packed=1), dict(variant=R.SMALL, rows_per_lane=2),
                dict(variant=R.SMALL, lanes_per_row=3)):
        assert f(X, Y, 64, 64, R.BF16, R.BF16, 0.5, 4, 0, 0, R.RowsmConfig(**cfg)) == R.EINVAL


def test_select_regimes(lib):
    s = R.rowsm_select
    d = lambda rows, cols, i, o, v=R.AUTO: R.rowsm_describe(rows, cols, i, o, v)
    # row of <= 32 vectors -> SMALL
    assert s(262144, 64, R.BF16, R.BF16) == R.SMALL
    assert s(10, 256, R.BF16, R.BF16) == R.SMALL      # 32 bf16 vectors of 8
    assert s(10, 257, R.BF16, R.BF16) == R.SMALL      # odd: the flat form
    assert s(10, 264, R.BF16, R.BF16) == R.MEDIUM     # 33 vectors
    assert s(10, 128, R.F32, R.F32) == R.SMALL
    assert s(10, 132, R.F32, R.F32) == R.MEDIUM
    assert s(10, 32, R.F32, R.F32) == R.SMALL
    # odd widths of 9-480 columns (narrow vectors of at most 4 bytes): the
    # flat form of the small family; 3-8 columns keep the packed small rows,
    # half-width vectors (60 bf16 columns) their plan
    for cols, i, o in ((33, R.F32, R.F32), (9, R.BF16, R.BF16), (77, R.BF16, R.F32),
                       (255, R.F32, R.BF16), (42, R.BF16, R.BF16)):
        t = d(10, cols, i, o)[1]
        assert t.startswith("small") and "flat=1 " in t and "block=64 " in t, t
    for cols, i, o in ((7, R.BF16, R.BF16), (481, R.F32, R.F32), (60, R.BF16, R.BF16),
                       (100, R.BF16, R.BF16)):
        assert "flat=0 " in d(10, cols, i, o)[1], (cols, d(10, cols, i, o)[1])
    # medium holds up to 16 waves x 64 lanes x 64 fp32 values (forced)
    d = lambda rows, cols, i, o, v=R.AUTO: R.rowsm_describe(rows, cols, i, o, v)
    assert s(64, 1000, R.F32, R.F32) == R.MEDIUM
    assert s(32768, 4096, R.BF16, R.BF16) == R.MEDIUM
    assert d(100, 65536, R.F32, R.F32, R.MEDIUM)[0] == R.OK
    assert d(100, 65540, R.F32, R.F32, R.MEDIUM)[0] == R.EINVAL
    assert s(100, 65540, R.F32, R.F32) == R.LARGE
    # packed bf16 rows up to 16 x 64 x 24 vectors of 8 (bf16 -> bf16 only:
    # bf16 -> f32 uses 4-element vectors so that each store is 16 bytes)
    assert "packed=1" in d(100, 196608, R.BF16, R.BF16, R.MEDIUM)[1]
    assert d(100, 196616, R.BF16, R.BF16, R.MEDIUM)[0] == R.EINVAL
    assert s(100, 196616, R.BF16, R.BF16) == R.LARGE
    assert s(4096, 151936, R.BF16, R.F32) == R.LARGE
    # rows of at least 64 KiB that need all 16 waves of a block: the split
    # form for rows of 80 KiB or more, shorter ones below cus / 2 or from
    # 8 cus rows (256 compute units)
    assert s(2047, 16384, R.F32, R.F32) == R.MEDIUM       # 64 KiB
    assert s(128, 16384, R.F32, R.F32) == R.MEDIUM
    assert s(127, 16384, R.F32, R.F32) == R.LARGE
    assert s(2048, 16384, R.F32, R.F32) == R.LARGE
    assert s(300, 32768, R.BF16, R.BF16) == R.MEDIUM      # 64 KiB
    assert s(300, 40960, R.BF16, R.BF16) == R.LARGE       # 80 KiB
    assert s(2047, 32768, R.F32, R.F32) == R.LARGE        # 128 KiB
    assert s(2048, 32768, R.F32, R.F32) == R.LARGE
    assert "split=4 " in d(2048, 32768, R.F32, R.F32)[1]     # ~128 bytes per lane
    assert s(100, 151936, R.BF16, R.BF16) == R.LARGE      # packed
    for rows, cols, dt in ((2047, 16384, R.F32), (300, 40960, R.BF16)):  # 16 waves
        assert "wpr=16 " in d(rows, cols, dt, dt, R.MEDIUM)[1]
    # full launches (>= 32 rows per compute unit) of rows of 129-4096 full
    # vectors take the measured shapes: two vectors per lane in the medium
    # form, the single-read form with 512 threads per row beyond
    def has(text, *parts):
        return all(p in text for p in parts)
    assert has(d(100000, 1024, R.F32, R.F32)[1], "medium", "wpr=2 ", "vpl=2 ", "block=128 ")
    assert has(d(100000, 2048, R.F32, R.F32)[1], "medium", "wpr=4 ", "vpl=2 ", "block=512 ")
    assert has(d(100000, 2048, R.BF16, R.F32)[1], "medium", "wpr=4 ", "vpl=2 ", "block=256 ")
    assert has(d(100000, 3072, R.BF16, R.F32)[1], "medium", "wpr=4 ", "vpl=3 ", "block=512 ")
    assert has(d(100000, 3072, R.F32, R.BF16)[1], "medium", "wpr=4 ", "vpl=3 ", "block=256 ")
    assert has(d(100000, 4096, R.F32, R.F32)[1], "medium", "wpr=8 ", "vpl=2 ", "block=512 ")
    assert has(d(32768, 4096, R.BF16, R.BF16)[1], "medium", "wpr=4 ", "vpl=2 ", "block=512 ")
    assert has(d(100000, 6144, R.F32, R.F32)[1], "large", "split=1 ", "block=512 ")
    assert has(d(100000, 6144, R.BF16, R.F32)[1], "medium", "wpr=8 ", "vpl=3 ")
    assert has(d(100000, 8192, R.F32, R.F32)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 8192, R.BF16, R.F32)[1], "large", "split=1 ", "block=512 ")
    assert has(d(100000, 8192, R.F32, R.BF16)[1], "large", "split=1 ", "block=512 ")
    assert has(d(100000, 16384, R.BF16, R.BF16)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 15360, R.BF16, R.BF16)[1], "large", "split=1 ", "block=512 ")
    assert has(d(100000, 20480, R.BF16, R.BF16)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 12288, R.F32, R.F32)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 14336, R.F32, R.F32)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 16384, R.F32, R.F32)[1], "large", "split=2 ", "block=512 ")
    assert has(d(100000, 16384, R.BF16, R.F32)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 11264, R.BF16, R.F32)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 9728, R.BF16, R.F32)[1], "large", "split=1 ", "block=512 ")
    assert has(d(100000, 9732, R.BF16, R.F32)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 18436, R.BF16, R.F32)[1], "large", "split=2 ", "block=512 ")
    assert has(d(100000, 16384, R.BF16, R.BF16)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 32768, R.BF16, R.BF16)[1], "large", "split=4 ", "block=256 ")
    # 4-16 rows per compute unit: the fewest waves per row that keep about two
    # 512-thread blocks per compute unit (at least what the registers need)
    assert has(d(1024, 8192, R.BF16, R.BF16)[1], "medium", "wpr=4 ", "vpl=4 ", "block=512 ")
    assert has(d(2048, 12288, R.BF16, R.BF16)[1], "medium", "wpr=2 ", "packed=1 ", "block=512 ")
    assert has(d(2048, 4096, R.F32, R.F32)[1], "medium", "wpr=2 ", "vpl=8 ", "block=512 ")
    assert has(d(4095, 8192, R.F32, R.F32)[1], "medium", "wpr=2 ", "vpl=16 ")
    assert has(d(4096, 4096, R.F32, R.F32)[1], "medium", "wpr=4 ", "vpl=4 ")   # the rule below
    assert has(d(1023, 4096, R.F32, R.F32)[1], "medium", "wpr=4 ", "vpl=4 ")
    assert has(d(2048, 16384, R.F32, R.F32)[1], "large")                      # 64 KiB rows
    # not below 32 rows per compute unit, nor for misaligned rows, forced
    # shapes or the fused form
    assert has(d(8191, 8192, R.F32, R.F32)[1], "medium", "wpr=8 ", "vpl=4 ")
    assert has(d(8192, 8192, R.F32, R.F32)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 8190, R.F32, R.F32)[1], "medium", "vw=4 ", "ragged=1 ",  # ragged:
               "wpr=4 ", "block=256 ")                                            # a row a block
    # ragged rows longer than one block's narrow vectors: from cus / 4 rows,
    # up to 16 waves of 10 fp32-width slots
    assert has(d(96, 30001, R.F32, R.F32)[1], "medium", "ragged=1 ", "wpr=16 ", "nv=8 ")
    assert has(d(32, 30001, R.F32, R.F32)[1], "large", "vw=1 ")
    assert has(d(200, 38401, R.F32, R.F32)[1], "medium", "ragged=1 ", "wpr=16 ", "nv=10 ")
    assert has(d(64, 16385, R.BF16, R.BF16)[1], "medium", "ragged=1 ")
    assert has(d(63, 16385, R.BF16, R.BF16)[1], "large", "vw=1 ")
    # the 4-16 rows per compute unit rule keeps the packed form up to 8 rows
    # per compute unit
    assert has(d(3656, 18520, R.BF16, R.BF16)[1], "medium", "wpr=8 ", "vpl=5 ", "packed=0 ")
    # rows under 64 KiB that the 16-value rule puts on 16 waves, outside the
    # row counts of the measured shapes and of the 4-16 rows per compute unit
    # rule: the fewest waves holding at most 48 values
    assert has(d(4096, 11984, R.BF16, R.BF16)[1], "medium", "wpr=4 ", "vpl=6 ", "packed=0 ")
    assert has(d(6144, 8240, R.BF16, R.F32)[1], "medium", "wpr=4 ", "vpl=9 ")
    assert has(d(768, 9920, R.F32, R.F32)[1], "medium", "wpr=4 ", "vpl=10 ")
    assert has(d(2048, 11984, R.BF16, R.BF16)[1], "medium", "wpr=2 ", "packed=1 ")  # 4-16 rule
    t = R.rowsm_describe_op(R.OP_SOFTMAX, 4096, 11984, R.BF16, R.BF16,
                            R.RowsmConfig(waves_per_row=16))[1]
    assert has(t, "medium", "wpr=16 ", "vpl=2 ")                                     # asked for
    t = R.rowsm_describe_op(R.OP_SOFTMAX, 100000, 8192, R.F32, R.F32,
                            R.RowsmConfig(waves_per_row=8))[1]
    assert has(t, "medium", "wpr=8 ", "vpl=4 ")
    t = R.rowsm_describe_op(R.OP_SCALED_CAUSAL, 100000, 2048, R.F32, R.BF16)[1]
    assert has(t, "medium", "wpr=1 ", "vpl=8 ")  # fused, bf16 out: 32 values per lane
    # the fused form with fp32 output has a table of its own
    fd = lambda cols, i: R.rowsm_describe_op(R.OP_SCALED_CAUSAL, 100000, cols, i, R.F32)[1]
    assert has(fd(1024, R.F32), "medium", "wpr=2 ", "vpl=2 ", "block=128 ")
    assert has(fd(4096, R.F32), "medium", "wpr=4 ", "vpl=4 ", "block=256 ")
    assert has(fd(12288, R.F32), "medium", "wpr=16 ", "vpl=3 ")
    assert has(fd(16384, R.F32), "large", "split=2 ", "block=256 ")
    assert has(fd(1024, R.BF16), "medium", "wpr=2 ", "block=256 ")
    assert has(fd(2048, R.BF16), "medium", "wpr=2 ", "vpl=4 ", "block=128 ")
    assert has(fd(5120, R.BF16), "medium", "wpr=4 ", "vpl=5 ")
    assert has(d(100000, 24576, R.BF16, R.BF16)[1], "large", "split=2 ", "block=256 ")
    assert has(d(100000, 18432, R.BF16, R.BF16)[1], "large", "split=2 ", "block=256 ")
    assert has(d(10000, 24576, R.BF16, R.F32)[1], "large", "split=2 ", "block=512 ")
    assert has(d(10000, 36864, R.BF16, R.F32)[1], "large", "split=4 ")  # beyond 8192 vectors
    # a single-read pick only while one group of blocks per row fits the
    # 2^20-block exchange workspace
    assert has(d(524288, 12288, R.F32, R.F32)[1], "large", "split=2 ")
    assert has(d(524289, 12288, R.F32, R.F32)[1], "medium", "wpr=16 ", "vpl=3 ")
    assert has(R.rowsm_describe_op(R.OP_LOG_SOFTMAX, 100000, 8192, R.F32, R.F32)[1],
               "large", "split=2 ", "block=256 ")
    bd = lambda rows, cols, i, o: R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, i, o)[1]
    assert bd(1023, 16384, R.F32, R.F32).startswith("medium")  # backward: from 4 cus rows
    assert bd(1024, 16384, R.F32, R.F32).startswith("large")
    assert "split=8 " in bd(1024, 16384, R.F32, R.F32) and "block=256" in bd(1024, 16384, R.F32, R.F32)
    assert bd(4096, 8192, R.F32, R.F32).startswith("medium")   # 32 KiB rows: unchanged
    assert "wpr=16 " in bd(4096, 8192, R.F32, R.F32)
    # backward launches of 4-16 rows per compute unit: few waves per row
    assert "wpr=4 " in bd(1024, 8192, R.F32, R.F32) and "vpl=8 " in bd(1024, 8192, R.F32, R.F32)
    assert "wpr=2 " in bd(2048, 6144, R.BF16, R.F32) and "vpl=12 " in bd(2048, 6144, R.BF16, R.F32)
    assert "wpr=16 " in bd(1023, 8192, R.F32, R.F32)
    # few long rows (>= 384 KiB of traffic): the split form fills the device
    # (the select assumes 256 compute units)
    assert s(63, 65536, R.F32, R.F32) == R.LARGE
    assert s(64, 65536, R.F32, R.F32) == R.LARGE          # and 64 values per lane
    assert s(64, 151936, R.BF16, R.BF16) == R.LARGE
    assert s(8, 32768, R.F32, R.F32) == R.LARGE           # 128 KiB rows, few: split
    assert s(8, 8192, R.F32, R.F32) == R.MEDIUM           # 32 KiB rows
    assert s(1024, 262144, R.F32, R.F32) == R.LARGE
    assert s(0, 5, R.F32, R.F32) > 0
    assert s(5, 5, 3, R.F32) == R.EDTYPE
    assert s(-5, 5, R.F32, R.F32) == R.EINVAL


def test_describe(lib):
    st, text = R.rowsm_describe(262144, 64, R.BF16, R.BF16)
    assert st == R.OK and text.startswith("small") and "lpr=8" in text and "vw=8" in text
    # rows that fill their lanes in launches of at least 40 MiB: one-wave
    # blocks with one row group per lane for a dtype pair of one width,
    # 128-thread blocks with two for a widening or narrowing pair; otherwise
    # 256-thread blocks, 4 row groups
    assert "block=64 " in text and "rpl=1 " in text and "grid=32768 " in text
    for rows, cols, dt in [(1048576, 64, R.BF16), (163840, 64, R.BF16), (8388608, 16, R.F32)]:
        t = R.rowsm_describe(rows, cols, dt, dt)[1]
        assert "block=64 " in t and "rpl=1 " in t, t
    for rows, cols, di, do in [(262144, 64, R.BF16, R.F32), (109227, 64, R.F32, R.BF16),
                               (2796202, 16, R.BF16, R.F32)]:
        t = R.rowsm_describe(rows, cols, di, do)[1]
        assert "block=128 " in t and "rpl=2 " in t, t
    for rows, cols, di, do in [(131072, 64, R.BF16, R.BF16),     # 32 MiB
                               (163839, 64, R.BF16, R.BF16),     # one row under 40 MiB
                               (65536, 64, R.BF16, R.F32),       # 24 MiB
                               (262144, 48, R.BF16, R.BF16)]:    # lanes left idle
        t = R.rowsm_describe(rows, cols, di, do)[1]
        assert "block=256 " in t and "rpl=4 " in t, t
    t = R.rowsm_describe_op(R.OP_SCALED_CAUSAL, 262144, 64, R.BF16, R.BF16)[1]
    assert "block=256 " in t and "rpl=4 " in t, t                  # fused: 4 row groups
    t = R.rowsm_describe_op(R.OP_LOG_SOFTMAX, 393216, 16, R.F32, R.F32)[1]
    assert "block=64 " in t and "rpl=1 " in t, t
    t = R.rowsm_describe_op(R.OP_LOG_SOFTMAX, 262144, 64, R.BF16, R.F32)[1]
    assert "block=128 " in t and "rpl=2 " in t, t
    # with the family or a lane grouping forced, the default grouping stays
    t = R.rowsm_describe(1048576, 64, R.BF16, R.BF16, R.SMALL)[1]
    assert "block=256 " in t and "rpl=4 " in t, t
    t = R.rowsm_describe_op(R.OP_SOFTMAX, 1048576, 64, R.BF16, R.BF16,
                            R.RowsmConfig(rows_per_lane=4))[1]
    assert "block=256 " in t and "rpl=4 " in t, t
    # the largest row counts: no product of rows and row bytes is formed
    t = R.rowsm_describe((1 << 61) + 1, 1, R.F32, R.F32)[1]
    assert "block=64 " in t and "rpl=1 " in t, t
    # the backward: one-wave blocks from 96 MiB of its three streams on (no
    # upper bound), for rows that fill their lanes and nothing forced
    bt = lambda rows, cols, dt, cfg=None: R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols,
                                                              dt, dt, cfg)[1]
    for rows, cols, dt in [(262144, 64, R.BF16), (4194304, 32, R.BF16), (131072, 128, R.F32),
                           ((1 << 40), 64, R.F32)]:
        t = bt(rows, cols, dt)
        assert t.startswith("small") and "block=64 " in t and "rpl=1 " in t, t
    assert "grid=32768 " in bt(262144, 64, R.BF16)
    for rows, cols, dt, cfg in [(262143, 64, R.BF16, None),      # just under 96 MiB
                                (524288, 48, R.BF16, None),       # lanes left idle
                                (262144, 64, R.BF16, R.RowsmConfig(rows_per_lane=4)),
                                (262144, 64, R.BF16, R.RowsmConfig(variant=R.SMALL))]:
        t = bt(rows, cols, dt, cfg)
        assert "block=256 " in t and "rpl=4 " in t, t
    t = bt(262144, 64, R.BF16, R.RowsmConfig(block=128))
    assert "block=128 " in t and "rpl=4 " in t, t
    st, text = R.rowsm_describe(32768, 4096, R.BF16, R.BF16)
    assert st == R.OK and text.startswith("medium")
    st, text = R.rowsm_describe(128, 151936, R.BF16, R.BF16, R.MEDIUM)
    assert st == R.OK and "packed=1" in text and "vpl=19" in text and "wpr=16" in text
    st, text = R.rowsm_describe(4096, 151936, R.BF16, R.F32)
    assert st == R.OK and text.startswith("large") and "vw=4" in text and "split=8" in text
    assert "nv=10" in text and "block=512" in text
    st, text = R.rowsm_describe(1024, 262144, R.F32, R.F32, R.LARGE)
    assert st == R.OK and text.startswith("large") and "split=8" in text and "nv=16" in text
    assert "block=512" in text and "grid=8192" in text and "one group of blocks per row" in text
    # a grid cap gives one residency whose groups loop over the rows
    st, text = R.rowsm_describe_op(R.OP_SOFTMAX, 1024, 262144, R.F32, R.F32,
                                   R.RowsmConfig(blocks_per_cu=2))
    assert st == R.OK and "split=8" in text and "one residency" in text
    # small and medium grids: one task per wave / one row group per block at
    # any row count; blocks_per_cu caps them (the waves then stride)
    # (4M rows of 64 bf16 columns take one-wave blocks of one row group per
    # lane, forward and backward)
    # (131072 rows of 4096 bf16 columns: the forward's 4 waves per row with 2
    # rows per block, the backward's measured 8 waves per row)
    for op, grid, wpr, mgrid in ((R.OP_SOFTMAX, 524288, 4, 65536),
                                 (R.OP_SOFTMAX_BACKWARD, 524288, 8, 131072)):
        st, text = R.rowsm_describe_op(op, 4194304, 64, R.BF16, R.BF16)
        assert st == R.OK and text.startswith("small") and f"grid={grid} " in text, text
        st, text = R.rowsm_describe_op(op, 4194304, 64, R.BF16, R.BF16,
                                       R.RowsmConfig(blocks_per_cu=8))
        assert st == R.OK and "grid=2048 " in text, text
        st, text = R.rowsm_describe_op(op, 131072, 4096, R.BF16, R.BF16)
        assert st == R.OK and text.startswith("medium") and f"wpr={wpr} " in text, text
        assert "block=512" in text and f"grid={mgrid} " in text, text
        st, text = R.rowsm_describe_op(op, 131072, 4096, R.BF16, R.BF16,
                                       R.RowsmConfig(blocks_per_cu=64))
        assert st == R.OK and "grid=16384 " in text, text
    # one wave per row and one to four slots: about 32 KiB of traffic per
    # block, rows / (32768 // row bytes) blocks rounded to whole residencies
    # of 4 blocks per compute unit, rows of whole lines or not
    for rows, cols, i, o, grid in ((1000000, 74, R.F32, R.F32, 18432),    # 296-byte rows
                                   (500000, 156, R.BF16, R.BF16, 9216),
                                   (500000, 164, R.F32, R.F32, 20480),
                                   (500000, 168, R.F32, R.F32, 20480),
                                   (500000, 256, R.F32, R.BF16, 23552),    # whole lines
                                   (500000, 256, R.F32, R.F32, 31744),
                                   (500000, 512, R.BF16, R.BF16, 31744),
                                   (500000, 260, R.BF16, R.BF16, 16384),   # two slots
                                   (2000, 74, R.F32, R.F32, 250)):         # uncapped grid
        st, text = R.rowsm_describe(rows, cols, i, o)
        assert st == R.OK and "wpr=1 " in text and f"block=512 grid={grid} " in text, text
    st, text = R.rowsm_describe(20000, 74, R.F32, R.F32)                 # at least 4 per CU
    assert st == R.OK and "grid=1024 " in text, text
    st, text = R.rowsm_describe(500000, 302, R.F32, R.F32)              # three slots
    assert st == R.OK and "nv=3 " in text and "grid=38912 " in text, text
    st, text = R.rowsm_describe(500000, 602, R.F32, R.F32)              # 152 vectors: ragged,
    assert st == R.OK and "ragged=1 " in text and "grid=500000 " in text, text  # a row a block
    # small rows of narrow vectors whose stores cover parts of lines: about
    # 16 KiB per block, whole residencies of 8 blocks per compute unit; full
    # vectors keep their rules
    st, text = R.rowsm_describe(1048576, 20, R.BF16, R.BF16)            # 80-byte rows
    assert st == R.OK and text.startswith("small") and "grid=6144 " in text, text
    st, text = R.rowsm_describe(1048576, 24, R.F32, R.F32)              # full vectors
    assert st == R.OK and text.startswith("small") and "grid=8192 " in text, text
    st, text = R.rowsm_describe_op(R.OP_SOFTMAX, 1000000, 37, R.F32, R.F32,
                                   R.RowsmConfig(blocks_per_cu=16))
    assert st == R.OK and "grid=4096 " in text, text
    st, text = R.rowsm_describe_op(R.OP_SCALED_CAUSAL, 1000000, 37, R.F32, R.F32)
    assert st == R.OK and "grid=250000 " in text, text                    # fused: unchanged
    # 512 threads would leave fewer than 8 blocks to the row: 256
    st, text = R.rowsm_describe(1024, 131072, R.F32, R.F32)
    assert st == R.OK and "split=8" in text and "block=256" in text
    cfg_two_pass = R.RowsmConfig(variant=R.LARGE, split_blocks=-1)
    st = R.rowsm_forward_config(X, Y, 4, 8, 7, R.F32, 0, cfg_two_pass)
    assert st == R.EDTYPE
    st, text = R.rowsm_describe(4, 4096, R.F32, R.F32, R.SMALL)
    assert st == R.EINVAL and text.startswith("error")
    st, text = R.rowsm_describe(0, 4096, R.F32, R.F32)
    assert st == R.OK and "no launch" in text


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(R.RowsmError):
        R.lib(str(tmp_path / "missing.so"))


def test_log_softmax_argument_errors(lib):
    f = R.rowsm_log_softmax
    assert f(X, Y, 4, 8, 7, R.F32, 0) == R.EDTYPE
    assert f(X, Y, -4, 8, R.F32, R.F32, 0) == R.EINVAL
    assert f(0, Y, 4, 8, R.F32, R.F32, 0) == R.EINVAL
    assert f(X, X + 4, 4, 8, R.F32, R.F32, 0) == R.EINVAL        # partial overlap
    assert f(X, X, 4, 8, R.BF16, R.F32, 0) == R.EINVAL           # in place, dtype change
    assert f(0, 0, 0, 8, R.F32, R.F32, 0) == R.OK                # empty
    assert f(X, Y, 64, 64, R.F32, R.F32, 0, R.RowsmConfig(variant=R.SMALL,
                                                         lanes_per_row=3)) == R.EINVAL
    # log-softmax takes the softmax plans
    for rows, cols, i, o in ((262144, 64, R.BF16, R.BF16), (64, 151936, R.BF16, R.BF16),
                             (4096, 151936, R.BF16, R.F32), (1024, 262144, R.F32, R.F32)):
        a = R.rowsm_describe_op(R.OP_LOG_SOFTMAX, rows, cols, i, o)
        b = R.rowsm_describe_op(R.OP_SOFTMAX, rows, cols, i, o)
        assert a == b and a[0] == R.OK


def test_backward_argument_errors(lib):
    f = R.rowsm_softmax_backward
    D = 0x7f4000000000                                             # a third fake buffer
    assert f(X, Y, D, 4, 8, 7, R.F32, 0) == R.EDTYPE
    assert f(X, Y, D, 4, 8, R.F32, 5, 0) == R.EDTYPE
    assert f(X, Y, D, -1, 8, R.F32, R.F32, 0) == R.EINVAL
    assert f(0, Y, D, 4, 8, R.F32, R.F32, 0) == R.EINVAL
    assert f(X, 0, D, 4, 8, R.F32, R.F32, 0) == R.EINVAL
    assert f(X, Y, 0, 4, 8, R.F32, R.F32, 0) == R.EINVAL
    assert f(X, Y, X + 4, 4, 8, R.F32, R.F32, 0) == R.EINVAL       # dx partially over y
    assert f(X, Y, Y + 4, 4, 8, R.F32, R.F32, 0) == R.EINVAL       # dx partially over dy
    assert f(X, Y, Y, 4, 8, R.BF16, R.F32, 0) == R.EINVAL          # in place, dtype change
    assert f(X, Y, D, 1, 1 << 30, R.F32, R.F32, 0) == R.EINVAL     # row too long
    assert f(0, 0, 0, 0, 8, R.F32, R.F32, 0) == R.OK               # empty: no launch
    assert f(X, Y, D, 64, 64, R.F32, R.F32, 0, R.RowsmConfig(packed=1)) == R.EINVAL
    assert f(X, Y, D, 64, 4096, R.F32, R.F32, 0, R.RowsmConfig(variant=R.SMALL)) == R.EINVAL
    assert f(X, Y, D, 64, 64, R.F32, R.F32, 0, R.RowsmConfig(variant=R.LARGE,
                                                             split_blocks=65)) == R.EINVAL


def test_backward_plans(lib):
    d = lambda rows, cols, i, o, **cfg: R.rowsm_describe_op(
        R.OP_SOFTMAX_BACKWARD, rows, cols, i, o, R.RowsmConfig(**cfg) if cfg else None)
    st, t = d(262144, 64, R.BF16, R.BF16)
    assert st == R.OK and t.startswith("small") and "lpr=8" in t and "rpl=1" in t  # 96 MiB
    # full launches (>= 32 rows per compute unit) of 129-4096 full vectors:
    # the measured backward shapes
    st, t = d(32768, 4096, R.BF16, R.BF16)                         # 512 vectors
    assert st == R.OK and t.startswith("medium") and "wpr=8 " in t and "nv=1 " in t, t
    st, t = d(8192, 4096, R.F32, R.F32)                            # 1024 vectors
    assert st == R.OK and t.startswith("large") and "split=1 " in t and "block=512" in t, t
    st, t = d(8192, 16384, R.F32, R.F32)                           # 4096 vectors
    assert st == R.OK and "split=2 " in t and "block=512" in t and "nv=4 " in t, t
    st, t = d(8192, 16384, R.F32, R.BF16)
    assert st == R.OK and "split=2 " in t and "block=512" in t and "nv=4 " in t, t
    st, t = d(8192, 16384, R.BF16, R.F32)                          # widening: medium
    assert st == R.OK and t.startswith("medium") and "wpr=16 " in t and "nv=4 " in t, t
    st, t = d(8192, 1024, R.BF16, R.BF16)                          # 128 vectors: not in it
    assert st == R.OK and "wpr=1 " in t and "nv=2 " in t, t
    # fewer rows, or a shape field given: the register-cap rule
    st, t = d(8191, 16384, R.F32, R.F32)
    assert st == R.OK and t.startswith("large") and "split=8 " in t, t
    st, t = d(32768, 4096, R.BF16, R.BF16, rows_per_block=2)
    assert st == R.OK and "wpr=4 " in t and "nv=2 " in t and "block=512" in t, t
    # medium holds at most 128 bytes of each input per lane: 16 x 64 x 8 vectors
    assert d(200, 65536, R.BF16, R.BF16)[1].startswith("medium")
    assert d(200, 65544, R.BF16, R.BF16)[1].startswith("large")
    assert d(200, 32768, R.F32, R.F32)[1].startswith("medium")
    # 16-wave rows of at least 64 KiB of each input in launches of fewer than
    # cus / 2 rows: the split form; from cus / 2 rows the medium form
    st, t = d(127, 16384, R.F32, R.F32)
    assert st == R.OK and t.startswith("large") and "split=8 " in t and "block=256" in t, t
    st, t = d(128, 16384, R.F32, R.F32)
    assert st == R.OK and t.startswith("medium") and "wpr=16 " in t, t
    assert d(127, 16380, R.F32, R.F32)[1].startswith("medium")     # under 64 KiB
    st, t = d(100, 65536, R.BF16, R.BF16, variant=R.MEDIUM)        # asked for
    assert st == R.OK and t.startswith("medium") and "wpr=16 " in t, t
    # rows of one wave and one to four slots: about 24 KiB of the three
    # streams per block, rows / (24576 // (cols * (2 ib + ob))) blocks in
    # whole residencies; five or more slots, small launches, a grid or a
    # shape given keep their plans
    cap = lambda rows, cols, dt, **cfg: int(d(rows, cols, dt, dt, **cfg)[1].split("grid=")[1].split()[0])
    assert cap(204600, 131, R.BF16) == 6144                       # 786-byte rows of 3 streams
    assert cap(291271, 90, R.F32) == 13312                        # 45 two-element vectors
    assert cap(204600, 300, R.BF16) == 15360                      # two slots
    assert cap(220289, 118, R.F32) == 13312
    assert cap(163840, 320, R.BF16) == 13312                      # 640-byte rows: whole lines
    assert cap(288070, 182, R.BF16) == 13312                      # three slots
    assert cap(288070, 330, R.BF16) == 36009                      # six: default grid
    assert cap(4000, 131, R.BF16) == 500                          # under the grid
    assert cap(204600, 131, R.BF16, blocks_per_cu=8) == 2048       # grid given
    assert cap(204600, 131, R.BF16, rows_per_block=4) == 51150     # shape given
    # few long rows (>= 512 KiB of y, dy and dx per row): the split form,
    # about one block per compute unit
    st, t = d(8, 65536, R.F32, R.F32)
    assert st == R.OK and t.startswith("large") and "split=32" in t
    st, t = d(4, 65536, R.BF16, R.BF16)                            # 384 KiB rows: the
    assert st == R.OK and t.startswith("large") and "split=16 " in t  # 16-wave redirect
    st, t = d(32, 151936, R.BF16, R.BF16)                          # register cap: 16
    assert st == R.OK and "split=16" in t and "nv=5" in t
    st, t = d(1024, 262144, R.F32, R.F32)
    assert st == R.OK and "split=16" in t and "nv=8" in t and "block=512" in t
    st, t = d(4, 64 * 256 * 8 * 4 + 4, R.F32, R.F32)                # 512-thread blocks
    assert st == R.OK and "split=33" in t and "block=512" in t
    # past 64 blocks x 512 threads x 8 vectors: the two-pass form
    st, t = d(4, 64 * 512 * 8 * 4 + 4, R.F32, R.F32)
    assert st == R.OK and "split=0" in t and "block=1024" in t
    assert d(4, 100, R.F32, R.F32, variant=R.MEDIUM, waves_per_row=16)[0] == R.OK
    assert d(4, 8, 9, R.F32)[0] == R.EDTYPE
    assert R.rowsm_describe_op(9, 4, 8, R.F32, R.F32)[0] == R.EINVAL


def test_moe_argument_errors_and_plans(lib):
    f = R.rowsm_moe_group_top2
    O = 0x7f4000000000
    assert f(X, O, 4, 64, 32, 7, R.F32, 0) == R.EDTYPE
    assert f(X, O, 4, 64, 32, R.F32, 3, 0) == R.EDTYPE
    for g in (0, 1, 3, 24, 128):
        assert f(X, O, 4, 64 * 3, g, R.F32, R.F32, 0) == R.EINVAL, g
    assert f(X, O, 4, 60, 32, R.F32, R.F32, 0) == R.EINVAL          # 32 does not divide 60
    assert f(X, O, -1, 64, 32, R.F32, R.F32, 0) == R.EINVAL
    assert f(0, O, 4, 64, 32, R.F32, R.F32, 0) == R.EINVAL
    assert f(X, 0, 4, 64, 32, R.F32, R.F32, 0) == R.EINVAL
    assert f(X, X + 256, 4, 64, 32, R.F32, R.F32, 0) == R.EINVAL    # output inside scores
    assert f(X, O + 2, 4, 64, 32, R.F32, R.F32, 0) == R.EINVAL      # misaligned f32 output
    assert f(X + 2, O, 4, 64, 32, R.F32, R.F32, 0) == R.EINVAL      # misaligned f32 scores
    assert f(0, 0, 0, 64, 32, R.F32, R.F32, 0) == R.OK              # empty: no launch
    assert f(X, O, 4, 64, 32, R.F32, R.F32, 0, R.RowsmConfig(variant=R.MEDIUM)) == R.EINVAL
    assert f(X, O, 4, 64, 32, R.F32, R.F32, 0, R.RowsmConfig(vw=8)) == R.EINVAL  # 32-byte vector
    d = lambda groups, g, i, **cfg: R.rowsm_describe_op(
        R.OP_MOE_GROUP_TOP2, groups, g, i, R.F32, R.RowsmConfig(**cfg) if cfg else None)
    st, t = d(1048576 * 8, 32, R.F32)
    assert st == R.OK and "vw=4" in t and "lpr=8" in t and "rpl=4" in t and "grid=65536" in t
    st, t = d(65536 * 8, 32, R.BF16)
    assert st == R.OK and "vw=8" in t and "lpr=4" in t
    st, t = d(1000, 2, R.F32)
    assert st == R.OK and "vw=2" in t and "lpr=1" in t
    st, t = d(100000 * 8, 32, R.F32, blocks_per_cu=1)
    assert st == R.OK and "grid=256" in t


def test_few_rows_split_counts(lib):
    # about one block per compute unit, at least 8 and at most 64 blocks per
    # row, at least two vectors per thread; never below the register minimum
    d = lambda rows, cols, i, o: R.rowsm_describe(rows, cols, i, o)[1]
    assert "split=32" in d(1, 65536, R.F32, R.F32) and "block=256" in d(1, 65536, R.F32, R.F32)
    assert "split=16" in d(16, 65536, R.F32, R.F32)
    assert "split=8" in d(32, 65536, R.F32, R.F32) and "split=8" in d(63, 65536, R.F32, R.F32)
    assert "split=64" in d(1, 262144, R.F32, R.F32)
    assert "split=32" in d(8, 262144, R.F32, R.F32)
    assert "split=8" in d(1024, 262144, R.F32, R.F32)               # many rows: registers
    assert "split=32" in d(8, 151936, R.BF16, R.F32) and "block=256" in d(8, 151936, R.BF16, R.F32)
    t = d(4096, 151936, R.BF16, R.F32)
    assert "split=8" in t and "block=512" in t                       # the vocab workload
    t = d(16, 262144, R.BF16, R.F32)
    assert "split=32" in t and "block=256" in t                      # raised to the register cap
    t = d(48, 262144, R.BF16, R.F32)
    assert "split=13" in t and "block=512" in t                      # 48 x 32 > 4 x 256 blocks
    t = d(128, 151936, R.F32, R.F32)
    assert "split=10" in t                                           # register plan


def test_stream_copy_argument_errors(lib):
    f = R.rowsm_stream_copy
    assert f(X, Y, 8, 7, R.F32, 0) == R.EDTYPE
    assert f(X, Y, 8, R.F32, 2, 0) == R.EDTYPE
    assert f(X, Y, -1, R.F32, R.F32, 0) == R.EINVAL
    assert f(X, Y, (1 << 60) + 1, R.F32, R.F32, 0) == R.EINVAL
    assert f(0, Y, 8, R.F32, R.F32, 0) == R.EINVAL
    assert f(X, 0, 8, R.F32, R.F32, 0) == R.EINVAL
    assert f(X + 2, Y, 8, R.F32, R.F32, 0) == R.EINVAL              # misaligned f32
    assert f(X, Y + 1, 8, R.F32, R.BF16, 0) == R.EINVAL             # misaligned bf16
    assert f(X, X + 16, 8, R.F32, R.F32, 0) == R.EINVAL             # partial overlap
    assert f(X, X, 8, R.BF16, R.F32, 0) == R.EINVAL                 # in place, widening
    assert f(X, X + 8, 8, R.BF16, R.F32, 0) == R.EINVAL             # output over the input
    assert f(0, 0, 0, R.F32, R.F32, 0) == R.OK                      # empty: no launch


def test_prefetch_config(lib):
    d = lambda rows, cols, i, o, **cfg: R.rowsm_describe_op(
        R.OP_SOFTMAX, rows, cols, i, o, R.RowsmConfig(**cfg))
    st, t = d(4096, 151936, R.BF16, R.F32, prefetch=1)
    assert st == R.OK and "prefetch=1" in t and "nv=10" in t
    assert d(1024, 262144, R.F32, R.F32, prefetch=1)[0] == R.EINVAL      # 64 values per lane
    assert d(1024, 262144, R.F32, R.F32, prefetch=1, split_blocks=32)[0] == R.OK
    assert d(8, 4096, R.F32, R.F32, prefetch=2)[0] == R.EINVAL            # outside its domain
    st, t = R.rowsm_describe_op(R.OP_SCALED_CAUSAL, 64, 262144, R.F32, R.F32,
                                R.RowsmConfig(prefetch=1, split_blocks=32))
    assert st == R.EINVAL                                                # fused: no prefetching


def test_backward_flat_plans():
    # odd widths of short rows: the flat form (flat_row.hpp) for 9-480
    # columns whose narrow vectors would be of at most 4 bytes, bf16 to bf16
    # only up to 128 columns (tiles of 2 vectors per lane where a row fits
    # them); asked for (small variant at the full vector width) up to what
    # one tile row holds; refused where the pointers are not aligned to the
    # full vector width
    def d(rows, cols, i, o, cfg=None):
        return R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, rows, cols, i, o, cfg)
    flat = lambda *a: "flat=1 " in d(*a)[1]
    assert flat(204600, 41, R.BF16, R.BF16) and flat(1000, 127, R.BF16, R.BF16)
    assert flat(204600, 21, R.BF16, R.BF16) and not flat(1000, 131, R.BF16, R.BF16)
    assert not flat(1000, 7, R.BF16, R.BF16) and flat(1000, 9, R.BF16, R.BF16)
    assert flat(1000, 21, R.F32, R.F32) and flat(1000, 479, R.F32, R.BF16)
    assert flat(1000, 9, R.BF16, R.F32) and not flat(1000, 7, R.BF16, R.F32)
    assert not flat(1000, 481, R.F32, R.F32) and not flat(1000, 90, R.F32, R.F32)
    assert not flat(1000, 44, R.BF16, R.BF16)                     # a multiple of 4
    st, t = d(1000, 41, R.BF16, R.BF16)
    assert t.startswith("small") and "vw=8 " in t and "lpr=8 " in t and "nv=8 " in t, t
    assert "rpl=2 " in t and "block=64 " in t, t
    assert "grid=" + str(-(-1000 // (1017 // 41))) + " " in t, t
    st, t = d(1000, 41, R.BF16, R.F32)                            # 4 vectors per lane
    assert "rpl=4 " in t and "grid=" + str(-(-1000 // (1021 // 41))) + " " in t, t
    cf = lambda vw: R.RowsmConfig(variant=R.SMALL, vw=vw)
    st, t = d(100, 1017, R.F32, R.F32, cf(4))
    assert st == R.OK and "flat=1 " in t and "lpr=64 " in t and "nv=16 " in t, t
    assert d(100, 1023, R.F32, R.F32, cf(4))[0] == R.EINVAL      # past one tile row
    st, t = d(100, 1023, R.BF16, R.BF16, cf(8))                 # past 2 vectors per lane
    assert st == R.OK and "rpl=4 " in t, t
    assert "rpl=2 " in d(100, 1017, R.BF16, R.BF16, cf(8))[1]
    assert d(100, 1025, R.BF16, R.BF16, cf(8))[0] == R.EINVAL    # past 1024
    assert "flat=1 " in d(10, 5, R.F32, R.F32, cf(4))[1]
    # vectors per lane of a tile through rows_per_lane: 4, or 2 for bf16 to
    # bf16 rows that fit such a tile (forward and backward)
    sl = lambda op, cols, i, o, vw, r: R.rowsm_describe_op(
        op, 1000, cols, i, o, R.RowsmConfig(variant=R.SMALL, vw=vw, rows_per_lane=r))
    for op in (R.OP_SOFTMAX, R.OP_LOG_SOFTMAX, R.OP_SOFTMAX_BACKWARD):
        assert "rpl=2 " in sl(op, 21, R.BF16, R.BF16, 8, 2)[1]
        assert "rpl=4 " in sl(op, 21, R.BF16, R.BF16, 8, 4)[1]
        assert "rpl=2 " in sl(op, 1017, R.BF16, R.BF16, 8, 2)[1]
        assert sl(op, 1023, R.BF16, R.BF16, 8, 2)[0] == R.EINVAL  # past 2 vectors
        assert sl(op, 21, R.F32, R.BF16, 4, 2)[0] == R.EINVAL     # bf16 pairs only
        assert sl(op, 21, R.BF16, R.BF16, 8, 1)[0] == R.EINVAL
        assert sl(op, 21, R.BF16, R.BF16, 8, 8)[0] == R.EINVAL
    # row phase: 4 lanes of 4 elements at 9-16 columns, else from 8 lanes;
    # lanes_per_row picks any compiled shape
    for op in (R.OP_SOFTMAX, R.OP_SOFTMAX_BACKWARD):
        for cols, lanes, e in ((9, 4, 4), (15, 4, 4), (17, 8, 4), (41, 8, 8), (255, 32, 8)):
            t = R.rowsm_describe_op(op, 1000, cols, R.F32, R.F32, None)[1]
            assert f"lpr={lanes} " in t and f"nv={e} " in t, (cols, t)
        lp = lambda cols, lanes: R.rowsm_describe_op(
            op, 1000, cols, R.F32, R.F32, R.RowsmConfig(variant=R.SMALL, vw=4, lanes_per_row=lanes))
        assert "lpr=8 " in lp(13, 8)[1] and "nv=2 " in lp(13, 8)[1]
        assert lp(21, 4)[0] == R.EINVAL                           # 4 x 8: not compiled
        assert lp(13, 2)[0] == R.EINVAL and lp(13, 1)[0] == R.EINVAL
        assert "lpr=8 " in lp(5, 0)[1]
    # the launcher: for bf16 to bf16, 2 up to 45 columns in the forward and
    # up to 128 in the backward; 4 otherwise
    au = lambda op, cols, i=R.BF16, o=R.BF16: R.rowsm_describe_op(op, 1000, cols, i, o, None)[1]
    for op in (R.OP_SOFTMAX, R.OP_LOG_SOFTMAX):
        assert "rpl=2 " in au(op, 21) and "rpl=2 " in au(op, 45) and "rpl=4 " in au(op, 47)
        assert "rpl=4 " in au(op, 77)
        assert "rpl=4 " in au(op, 21, R.F32, R.F32) and "rpl=4 " in au(op, 21, R.BF16, R.F32)
    assert "rpl=2 " in au(R.OP_SOFTMAX_BACKWARD, 127)
    assert "rpl=4 " in au(R.OP_SOFTMAX_BACKWARD, 21, R.F32, R.BF16)
    assert d(10, 64, R.F32, R.F32, R.RowsmConfig(variant=R.SMALL, vw=8))[0] == R.EINVAL
