"""bench.py's rocprofv3 summarisers on the CPU, with synthetic rocprofv3 CSV
output: dispatches are attributed to the launches of the bench JSON line by
kernel name, template arguments, workgroup and grid size; the launcher check's
in launch order; counters are scaled by the calibration copy."""
import csv
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
import bench_profiles as P  # noqa: E402

TRACE_COLS = ["Kind", "Agent_Id", "Queue_Id", "Stream_Id", "Thread_Id", "Dispatch_Id",
              "Kernel_Id", "Kernel_Name", "Correlation_Id", "Start_Timestamp", "End_Timestamp",
              "Private_Segment_Size", "Group_Segment_Size", "Workgroup_Size_X",
              "Workgroup_Size_Y", "Workgroup_Size_Z", "Grid_Size_X", "Grid_Size_Y",
              "Grid_Size_Z"]
PMC_COLS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id",
            "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size",
            "Scratch_Size", "VGPR_Count", "Accum_VGPR_Count", "SGPR_Count", "Counter_Name",
            "Counter_Value", "Start_Timestamp", "End_Timestamp"]

SMALL = "void rowsm::small_row_kernel<rowsm::BF16, rowsm::BF16, 8, 8, 1, 0>(x const*, y*, long, int, rowsm::Fused)"
SMALL_LOG = "void rowsm::small_row_kernel<rowsm::BF16, rowsm::BF16, 8, 8, 1, 2>(x const*, y*, long, int, rowsm::Fused)"
SPLIT = "void rowsm::split_row_kernel<rowsm::F32, rowsm::F32, 4, 16, 0, false>(x const*, y*, long, int, int, rowsm::SplitWorkspace, unsigned int, rowsm::Fused)"
COPY = "void rowsm::(anonymous namespace)::stream_copy_kernel<rowsm::F32, rowsm::F32, 4>(x const*, y*, long, long)"
FILL = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float>>(int, F, A)"

SMALL_DESC = ("small vw=8 nvec=8 lpr=8 rpl=1 wpr=1 vpl=1 nv=1 packed=0 u=4 split=0 stream=0 "
              "prefetch=0 block=64 grid=32768 (grid assumes 256 CUs)")
SPLIT_DESC = ("large vw=4 nvec=65536 lpr=1 rpl=4 wpr=1 vpl=16 nv=16 packed=0 u=4 split=8 "
              "stream=0 prefetch=0 block=512 grid=8192 (one group of blocks per row)")


def bench_line():
    return {"metric": bench.METRIC, "value": 6500.0, "ms_per_step": 1.0,
            "regimes_detail": {
                "small_262144x64": {"launch": SMALL_DESC, "algorithmic_bytes": 67108864,
                                    "avg_us": 15.0, "copy_us": 16.0},
                "large_1024x262144": {"launch": SPLIT_DESC,
                                      "algorithmic_bytes": 2147483648, "avg_us": 335.0,
                                      "copy_us": 340.0}}}


def write_trace(d, rows):
    os.makedirs(d / "host" / "123", exist_ok=True)
    with open(d / "host" / "123" / "123_bench_kernel_trace.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=TRACE_COLS)
        w.writeheader()
        t = 1000
        for i, (name, block, grid, us) in enumerate(rows):
            w.writerow({"Kind": "KERNEL_DISPATCH", "Dispatch_Id": i + 1, "Kernel_Name": name,
                        "Start_Timestamp": t, "End_Timestamp": t + int(us * 1000),
                        "Workgroup_Size_X": block, "Workgroup_Size_Y": 1,
                        "Workgroup_Size_Z": 1, "Grid_Size_X": grid, "Grid_Size_Y": 1,
                        "Grid_Size_Z": 1})
            t += 1000000


def write_pmc(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(d / "1_pmc_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=PMC_COLS)
        w.writeheader()
        for i, (name, block, grid, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Workgroup_Size": block,
                        "Grid_Size": grid, "Counter_Name": counter, "Counter_Value": value})


def test_kernel_name_parsing():
    assert P.parse_kernel_name(SPLIT) == (
        "split_row_kernel", ["rowsm::F32", "rowsm::F32", "4", "16", "0", "false"])
    assert P.parse_kernel_name(COPY)[0] == "stream_copy_kernel"
    assert P.parse_kernel_name(FILL) == (None, [])


def test_launch_specs():
    s = P.launch_spec("softmax", SPLIT_DESC, "f32", "f32")
    assert s["base"] == "split_row_kernel" and s["block"] == 512 and s["grid"] == 512 * 8192
    assert s["args"][4] == "0" and s["args"][3] == "16"
    assert P.launch_spec("log_softmax", SPLIT_DESC, "f32", "f32")["args"][4] == "2"
    assert P.launch_spec("backward", SPLIT_DESC, "f32", "f32")["base"] == "bwd_split_kernel"
    two_pass = SPLIT_DESC.replace("split=8", "split=0")
    assert P.launch_spec("softmax", two_pass, "f32", "f32")["base"] == "large_row_kernel"
    assert P.launch_spec("moe", SMALL_DESC, "bf16", "f32")["base"] == "group_top2_kernel"
    ragged = ("medium vw=8 nvec=501 lpr=1 rpl=4 wpr=2 vpl=4 nv=4 packed=0 u=4 split=0 "
              "stream=0 prefetch=0 ragged=1 flat=0 block=128 grid=12288 (grid assumes 256 CUs)")
    r = P.launch_spec("log_softmax", ragged, "bf16", "bf16")
    assert r["base"] == "ragged_row_kernel" and r["args"][3] == "4" and r["args"][4] == "2"
    flat = ("small vw=8 nvec=11 lpr=16 rpl=4 wpr=1 vpl=8 nv=8 packed=0 u=4 split=0 stream=0 "
            "prefetch=0 ragged=0 flat=1 block=64 grid=80660 (grid assumes 256 CUs)")
    fl = P.launch_spec("softmax", flat, "bf16", "bf16")
    assert fl["base"] == "flat_row_kernel" and fl["block"] == 64 and fl["grid"] == 64 * 80660
    bf = P.launch_spec("backward", flat, "bf16", "bf16")
    assert bf["base"] == "bwd_flat_kernel" and bf["grid"] == 64 * 80660
    assert bf["args"] == {0: "rowsm::BF16", 1: "rowsm::BF16", 2: "8", 3: "16", 4: "8", 5: "4"}
    assert fl["args"][6] == "4"
    assert fl["args"][2] == "8" and fl["args"][3] == "16" and fl["args"][4] == "8"
    assert fl["args"][5] == "0"
    c = P.copy_spec(1024 * 262144, "f32", "f32")
    assert c["grid"] == 1024 * 262144 // 4 and c["args"][2] == "4"
    assert P.copy_spec(1000, "bf16", "f32")["grid"] == 256  # one partial block


def test_trace_summary(tmp_path):
    log = tmp_path / "bench.log"
    log.write_text("noise\n" + json.dumps(bench_line()) + "\n")
    write_trace(tmp_path / "trace", [
        (FILL, 256, 1 << 20, 100.0),
        (SMALL, 64, 2097152, 12.0), (SMALL, 64, 2097152, 14.0),
        (SMALL_LOG, 64, 2097152, 99.0),          # another output form: not the regime
        (SMALL, 256, 2097152, 99.0),             # another block size: not the regime
        (SPLIT, 512, 4194304, 330.0),
        (COPY, 256, 1024 * 262144 // 4, 336.0),
    ])
    text = P.summarize_trace(str(log), str(tmp_path / "trace"), "rocprofv3 ...", 8000.0)
    rows = {ln.split("|")[1].strip() + "/" + ln.split("|")[2].strip().split(" ")[0]: ln
            for ln in text.splitlines() if ln.startswith("| ") and "---" not in ln}
    small = rows["regimes/small_262144x64"].split("|")
    assert small[6].strip() == "2" and small[7].strip() == "13.00"
    large = rows["regimes/large_1024x262144"].split("|")
    assert large[6].strip() == "1" and large[7].strip() == "330.00"
    assert float(large[11]) == pytest.approx(2147483648 / 330e3, abs=1)
    assert rows["copy/large_1024x262144"].split("|")[6].strip() == "1"
    assert rows["copy/small_262144x64"].split("|")[6].strip() == "0"


def test_counter_summary(tmp_path):
    log = tmp_path / "bench.log"
    log.write_text(json.dumps(bench_line()) + "\n")
    cal = "__amd_rocclr_copyBuffer"
    write_pmc(tmp_path / "cf", "FETCH_SIZE", [(cal, 256, 1 << 26, 524288.0)] * 3)
    write_pmc(tmp_path / "cw", "WRITE_SIZE", [(cal, 256, 1 << 26, 1048576.0)] * 3)
    write_pmc(tmp_path / "f", "FETCH_SIZE", [(SMALL, 64, 2097152, 16400.0),
                                             (SPLIT, 512, 4194304, 526000.0)])
    write_pmc(tmp_path / "w", "WRITE_SIZE", [(SMALL, 64, 2097152, 32768.0),
                                             (SPLIT, 512, 4194304, 1048576.0)])
    text, table = P.summarize_counters(str(log), str(tmp_path / "f"), str(tmp_path / "w"),
                                       str(tmp_path / "cf"), str(tmp_path / "cw"), 1 << 30,
                                       "cmds", bench.kernel_source_hash, bench.kernel_family)
    assert table["fetch_scale"] == pytest.approx(2.0) and table["write_scale"] == 1.0
    s = table["launches"]["small_262144x64"]
    assert s["fetch_bytes"] == pytest.approx(16400 * 1024 * 2.0)
    assert s["fetch_over_input_bytes"] == pytest.approx(16400 * 2048 / 33554432)
    assert s["write_over_output_bytes"] == pytest.approx(1.0)
    assert s["source_hash"] == bench.kernel_source_hash("small_row")
    assert s["launch"] == SMALL_DESC
    big = table["launches"]["large_1024x262144"]
    assert big["hbm_bytes_per_launch"] == pytest.approx(big["fetch_bytes"] + big["write_bytes"])
    # the table is what bench.py's measured_traffic() reads
    p = tmp_path / "t.json"
    p.write_text(json.dumps(table))
    old = bench.PROFILE_COUNTERS
    try:
        bench.PROFILE_COUNTERS = str(p)
        assert bench.measured_traffic("small_262144x64", SMALL_DESC) == s["hbm_bytes_per_launch"]
    finally:
        bench.PROFILE_COUNTERS = old


def test_launcher_summary_in_launch_order(tmp_path):
    res = {"reps_per_shape": 3, "launcher_check": [
        {"op": "softmax", "rows": 262144, "cols": 64, "in": "bf16", "out": "bf16",
         "launch": SMALL_DESC, "timed": ["auto", "b256r4"], "us": {}}]}
    log = tmp_path / "lc.log"
    log.write_text(json.dumps(res) + "\n")
    rows = [(SMALL, 64, 2097152, 50.0), (FILL, 256, 1 << 20, 9.0), (SMALL, 64, 2097152, 12.0),
            (SMALL, 64, 2097152, 12.0)]
    rows += [(SMALL.replace("8, 8, 1, 0", "8, 8, 4, 0"), 256, 524288, u) for u in (9, 13, 13)]
    write_trace(tmp_path / "t", rows)
    text = P.summarize_launcher(str(log), str(tmp_path / "t"), "cmd", 8000.0)
    line = [ln for ln in text.splitlines() if ln.startswith("| softmax")][0].split("|")
    assert line[5].strip() == "12.0" and line[6].strip() == "auto"
    # a trace whose dispatch count does not fit the check's launches is refused
    write_trace(tmp_path / "t2", rows[:-1])
    with pytest.raises(ValueError):
        P.summarize_launcher(str(log), str(tmp_path / "t2"), "cmd", 8000.0)


def test_parity_gate_rows_and_planted_error():
    import torch

    from paper_2607_23089_amd import workloads as W
    rows = bench.gate_rows(32768)
    assert rows[0] == 0 and rows[-1] == 32767
    assert len(rows) <= 32 and rows == sorted(set(rows))
    assert bench.gate_rows(3) == [0, 1, 2]
    w = W.WORKLOADS["fp32_64x1000"]
    x = W.make_input(w)
    y = torch.softmax(x.double(), dim=-1).float()
    ok = bench.parity_gate({w.name: x}, {w.name: y}, [w.name], threads=2)
    assert ok[w.name]["parity_ok"] and ok[w.name]["rows_checked"] == len(bench.gate_rows(64))
    y[bench.gate_rows(64)[5], 17] += 1e-5       # a planted error on a gated row
    bad = bench.parity_gate({w.name: x}, {w.name: y}, [w.name], threads=2)
    assert not bad[w.name]["parity_ok"]


def test_size_sweep_summary_fits_fixed_cost_and_rate(tmp_path):
    # two sizes of at least 64 MiB whose durations lie on 1 us + bytes / 6400 GB/s
    sizes = [(1048576, 256, 2097152), (2097152, 256, 4194304)]
    res = {"launches_per_size": 3, "size_sweep": []}
    rows = []
    for r, blk, grid_threads in sizes:
        nbytes = r * 64 * 4
        desc = SMALL_DESC.replace("block=64 grid=32768", f"block={blk} grid={grid_threads // blk}")
        res["size_sweep"].append({"rows": r, "cols": 64, "bytes": nbytes, "launch": desc,
                                  "avg_us": 0.0, "copy_us": 0.0})
        t = 1.0 + nbytes / 6400e3
        rows += [(SMALL, blk, grid_threads, 99.0)] + [(SMALL, blk, grid_threads, t)] * 2
        rows += [(COPY.replace("F32, rowsm::F32, 4", "BF16, rowsm::BF16, 8"), 256,
                  nbytes // 4 // 16 * 4, t + 0.5)] * 3
    log = tmp_path / "sweep.log"
    log.write_text(json.dumps(res) + "\n")
    write_trace(tmp_path / "t", rows)
    text = P.summarize_sweep(str(log), str(tmp_path / "t"), "cmd", 8000.0)
    fit = [ln for ln in text.splitlines() if ln.startswith("Least-squares")][0]
    assert "= 1.00 us + bytes / 6400 GB/s" in fit, fit
    write_trace(tmp_path / "t2", rows[:-1])
    with pytest.raises(ValueError):
        P.summarize_sweep(str(log), str(tmp_path / "t2"), "cmd", 8000.0)


def test_pmc_summary(tmp_path):
    log = tmp_path / "bench.log"
    log.write_text(json.dumps(bench_line()) + "\n")
    d = tmp_path / "pmc"
    write_pmc(d, "VALUBusy", [(SMALL, 64, 2097152, 20.0), (SMALL, 64, 2097152, 30.0)])
    text = P.summarize_pmc(str(log), str(d), "cmd")
    line = [ln for ln in text.splitlines() if ln.startswith("| regimes | small")][0]
    assert "| 2 | 25 |" in line


def test_overlap_summary(tmp_path):
    da = ("large vw=4 nvec=65536 lpr=1 rpl=4 wpr=1 vpl=16 nv=16 packed=0 u=4 split=16 "
          "stream=0 prefetch=0 block=256 grid=256 (one group of blocks per row)")
    db = ("large vw=4 nvec=37984 lpr=1 rpl=4 wpr=1 vpl=10 nv=10 packed=0 u=4 split=16 "
          "stream=0 prefetch=0 block=256 grid=512 (one group of blocks per row)")
    res = {"stream_overlap": {"launch_a": da, "launch_b": db, "pairs": 2,
                              "warm_up_launches": 2, "outputs_equal_to_launches_alone": True}}
    log = tmp_path / "ov.log"
    log.write_text(json.dumps(res) + "\n")
    A = "void rowsm::split_row_kernel<rowsm::F32, rowsm::F32, 4, 16, 0, false>(...)"
    B = "void rowsm::split_row_kernel<rowsm::BF16, rowsm::F32, 4, 10, 0, false>(...)"
    d = tmp_path / "t" / "h" / "1"
    os.makedirs(d)
    rows = [(A, 256, 65536, 0, 10), (B, 256, 131072, 20, 30),        # references, alone
            (A, 256, 65536, 40, 50), (B, 256, 131072, 60, 70),      # warm-up, one per stream
            (A, 256, 65536, 100, 110), (B, 256, 99999, 105, 115),   # half overlap
            (A, 256, 65536, 200, 210), (B, 256, 131072, 220, 230)]  # none
    with open(d / "1_t_kernel_trace.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=TRACE_COLS)
        w.writeheader()
        for i, (name, blk, grid, t0, t1) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Start_Timestamp": t0 * 1000,
                        "End_Timestamp": t1 * 1000, "Workgroup_Size_X": blk,
                        "Workgroup_Size_Y": 1, "Workgroup_Size_Z": 1, "Grid_Size_X": grid,
                        "Grid_Size_Y": 1, "Grid_Size_Z": 1})
    text = P.summarize_overlap(str(log), str(tmp_path / "t"), "cmd")
    # A at 100-110 shares 5 us with B at 105-115; A at 200-210 shares nothing
    assert "Both streams had a kernel running for 5.0 us of the 130.0 us" in text, text
    assert "2 of 4 launches ran partly alongside" in text, text
