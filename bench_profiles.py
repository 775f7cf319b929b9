"""rocprofv3 summaries for profiles/, written from the CSV output of rocprofv3
runs of bench.py (``bench.py --summarize-trace`` / ``--summarize-counters`` /
``--summarize-launcher``; no GPU needed).

Dispatches are attributed to the launches bench.py reports in its JSON line:
each launch's description (``rowsm_describe``: family, vector width, slot
count, single-read blocks per row, block and grid) and the operation of its
leg determine the kernel's name, template arguments, workgroup size and grid
size, which the dispatch must match.  Copies of the library's streaming copy
are matched by dtype pair and grid size.  The launcher check's dispatches are
taken in launch order: every timed shape makes a fixed number of launches.
"""
from __future__ import annotations

import csv
import glob
import json
import os
import re

# Kernels of the library (names without the namespace).
ROW_KERNELS = ("small_row_kernel", "medium_row_kernel", "split_row_kernel",
               "large_row_kernel", "ragged_row_kernel", "flat_row_kernel", "bwd_small_kernel",
               "bwd_flat_kernel", "bwd_medium_kernel",
               "bwd_split_kernel", "bwd_large_kernel", "group_top2_kernel",
               "stream_copy_kernel")
# Index of the output-form template argument (plain 0, fused 1, log 2).
MODE_ARG = {"small_row_kernel": 5, "medium_row_kernel": 5, "split_row_kernel": 4,
            "large_row_kernel": 4, "ragged_row_kernel": 4, "flat_row_kernel": 5}
MODES = {"softmax": 0, "scaled_causal": 1, "log_softmax": 2}
TYPE_NAMES = {"f32": "rowsm::F32", "bf16": "rowsm::BF16"}
DTYPE_BYTES = {"f32": 4, "bf16": 2}
COPY_BLOCK = 256  # threads per block of the streaming copy


# ---- reading rocprofv3 output ---------------------------------------------

def read_csv_rows(root: str, suffix: str) -> list:
    """Rows of every ``*<suffix>`` CSV file under root (rocprofv3 writes one per
    process, in subdirectories named for the host and process)."""
    rows = []
    for path in sorted(glob.glob(os.path.join(root, "**", "*" + suffix), recursive=True)):
        with open(path, newline="") as f:
            rows.extend(csv.DictReader(f))
    if not rows:
        raise FileNotFoundError(f"no *{suffix} under {root}")
    return rows


def _size(row: dict, base: str) -> int:
    if row.get(base) not in (None, ""):
        return int(float(row[base]))
    n = 1
    for ax in ("X", "Y", "Z"):
        v = row.get(f"{base}_{ax}")
        if v not in (None, ""):
            n *= int(float(v))
    return n


def parse_kernel_name(name: str):
    """('split_row_kernel', ['rowsm::BF16', 'rowsm::F32', '4', '10', '0', 'false'])
    from a demangled name such as 'void rowsm::split_row_kernel<rowsm::BF16,
    rowsm::F32, 4, 10, 0, false>(...)'; (None, []) for other kernels."""
    m = re.search(r"(?:rowsm::)?(\w+)<([^<>]*)>", name)
    if not m or m.group(1) not in ROW_KERNELS:
        return None, []
    return m.group(1), [a.strip() for a in m.group(2).split(",")]


def dispatches(rows: list) -> list:
    """Kernel-trace rows -> dicts with base, args, block, grid (threads),
    duration (us) and dispatch id, in dispatch order."""
    out = []
    for r in rows:
        base, args = parse_kernel_name(r.get("Kernel_Name", ""))
        out.append({"name": r.get("Kernel_Name", ""), "base": base, "args": args,
                    "block": _size(r, "Workgroup_Size"), "grid": _size(r, "Grid_Size"),
                    "us": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
                    if r.get("End_Timestamp") else None,
                    "id": int(r.get("Dispatch_Id") or 0), "row": r})
    out.sort(key=lambda d: d["id"])
    return out


# ---- what each reported launch looks like in a trace -------------------------

def parse_launch(desc: str) -> dict:
    """Fields of a launch description ('medium vw=8 ... block=512 grid=16384 ...')."""
    f = {"family": desc.split(" ", 1)[0]}
    for k, v in re.findall(r"(\w+)=(-?\d+)", desc):
        f[k] = int(v)
    return f


def launch_spec(op: str, desc: str, din: str, dout: str) -> dict:
    """Kernel base name, required template arguments, block and grid threads of
    the launch described by desc for operation op."""
    f = parse_launch(desc)
    fam = f["family"]
    if op == "moe":
        base = "group_top2_kernel"
    elif op == "backward":
        base = {"small": "bwd_small_kernel", "medium": "bwd_medium_kernel"}.get(fam) or \
            ("bwd_split_kernel" if f.get("split", 0) > 0 else "bwd_large_kernel")
        if base == "bwd_small_kernel" and f.get("flat", 0):
            base = "bwd_flat_kernel"
    else:
        base = {"small": "small_row_kernel", "medium": "medium_row_kernel"}.get(fam) or \
            ("split_row_kernel" if f.get("split", 0) > 0 else "large_row_kernel")
        if base == "medium_row_kernel" and f.get("ragged", 0):
            base = "ragged_row_kernel"
        if base == "small_row_kernel" and f.get("flat", 0):
            base = "flat_row_kernel"
    args = {0: TYPE_NAMES[din], 1: TYPE_NAMES[dout], 2: str(f["vw"])}
    if base in MODE_ARG:
        args[MODE_ARG[base]] = str(MODES[op])
    if base in ("medium_row_kernel", "split_row_kernel", "ragged_row_kernel") or \
            base in ("bwd_medium_kernel", "bwd_split_kernel"):
        args[3] = str(f["nv"])
    if base in ("flat_row_kernel", "bwd_flat_kernel"):  # lanes per row and elements per lane of the row phase
        args[3] = str(f["lpr"])
        args[4] = str(f["nv"])
        # vectors per lane of a tile
        args[6 if base == "flat_row_kernel" else 5] = str(f["rpl"])
    return {"base": base, "args": args, "block": f["block"], "grid": f["block"] * f["grid"]}


def copy_spec(n: int, din: str, dout: str) -> dict:
    """The streaming copy of n elements: one vector of at most 16 bytes (input
    and output side) per thread, blocks of 256 threads."""
    vw = 16 // max(DTYPE_BYTES[din], DTYPE_BYTES[dout])
    blocks = -(-n // (vw * COPY_BLOCK))
    return {"base": "stream_copy_kernel",
            "args": {0: TYPE_NAMES[din], 1: TYPE_NAMES[dout], 2: str(vw)},
            "block": COPY_BLOCK, "grid": blocks * COPY_BLOCK}


def matches(spec: dict, d: dict) -> bool:
    if d["base"] != spec["base"] or d["block"] != spec["block"] or d["grid"] != spec["grid"]:
        return False
    return all(i < len(d["args"]) and d["args"][i] == v for i, v in spec["args"].items())


def bench_targets(res: dict) -> list:
    """(row, workload, spec, algorithmic bytes, HIP-event us, traffic key) for
    every launch the bench JSON line reports."""
    from paper_2607_23089_amd import workloads as W

    t = []
    for name, p in res.get("regimes_detail", {}).items():
        w = W.WORKLOADS[name]
        t.append(("regimes", name, launch_spec("softmax", p["launch"], w.in_dtype, w.out_dtype),
                  p["algorithmic_bytes"], p["avg_us"], name))
    for name, p in res.get("regimes_detail", {}).items():
        w = W.WORKLOADS[name]
        t.append(("copy", name, copy_spec(w.rows * w.cols, w.in_dtype, w.out_dtype),
                  p["algorithmic_bytes"], p.get("copy_us"), f"copy/{name}"))
    nxt = res.get("next_rows", {})
    fz = nxt.get("fused_scale_causal")
    if fz and "launch" in fz:
        t.append(("fused", "causal_32768x4096",
                  launch_spec("scaled_causal", fz["launch"], "bf16", "bf16"),
                  fz["algorithmic_bytes"], fz["avg_us"], "fused/causal_32768x4096"))
        if "copy_elements" in fz:
            t.append(("fused copy", "causal_32768x4096",
                      copy_spec(fz["copy_elements"], "bf16", "f32"),
                      fz["copy_elements"] * 6, fz.get("copy_1to2_us"),
                      "fused_copy/causal_32768x4096"))
    for name, p in nxt.get("log_softmax", {}).items():
        w = W.WORKLOADS[name]
        t.append(("log_softmax", name, launch_spec("log_softmax", p["launch"], w.in_dtype,
                                                   w.out_dtype),
                  p["algorithmic_bytes"], p["avg_us"], f"log_softmax/{name}"))
    for name, p in nxt.get("softmax_backward", {}).items():
        w = W.BACKWARD_WORKLOADS[name]
        t.append(("softmax_backward", name, launch_spec("backward", p["launch"], w.in_dtype,
                                                        w.out_dtype),
                  p["algorithmic_bytes"], p["avg_us"], f"softmax_backward/{name}"))
    for name, p in nxt.get("moe_group_top2", {}).items():
        w = W.MOE_WORKLOADS[name]
        t.append(("moe_group_top2", name, launch_spec("moe", p["launch"], w.in_dtype,
                                                      w.out_dtype),
                  p["algorithmic_bytes"], p["avg_us"], f"moe_group_top2/{name}"))
    lb = res.get("launch_bound")
    if lb:
        t.append(("launch_bound", "fp32_64x1000", launch_spec("softmax", lb["launch"], "f32",
                                                              "f32"),
                  W.WORKLOADS["fp32_64x1000"].algorithmic_bytes, lb.get("median_us_alone"),
                  "fp32_64x1000"))
    return t


def attribute(targets: list, ds: list) -> list:
    """Dispatches of each target.  Targets with the same kernel, template
    arguments, block and grid share their dispatches (e.g. the copies of the
    same bytes in two legs); such rows say so."""
    out = []
    for tg in targets:
        got = [d for d in ds if matches(tg[2], d)]
        shared = [o[0] + " " + o[1] for o in targets
                  if o is not tg and o[2] == tg[2]]
        out.append((tg, got, shared))
    return out


def read_bench_json(path: str) -> dict:
    """The last JSON line bench.py printed into a log."""
    line = None
    with open(path) as f:
        for ln in f:
            if ln.startswith("{"):
                line = ln
    if line is None:
        raise ValueError(f"no JSON line in {path}")
    return json.loads(line)


def _short(name: str) -> str:
    base, args = parse_kernel_name(name)
    return f"{base}<{', '.join(args)}>" if base else name


# ---- summaries ------------------------------------------------------------

def summarize_trace(bench_log: str, trace_dir: str, command: str, peak_gbs: float) -> str:
    res = read_bench_json(bench_log)
    ds = dispatches(read_csv_rows(trace_dir, "kernel_trace.csv"))
    lines = [
        "# Kernel trace: row-softmax regimes and the next rows (bench.py default run)",
        "",
        "Command (repository root, MI355X):",
        "",
        "    " + command.replace("\n", "\n    "),
        "",
        "Written by `python3 bench.py --summarize-trace` from that run's kernel trace "
        "(`*kernel_trace.csv`) and the JSON line it printed.  Each launch the JSON line "
        "reports is matched to its dispatches by kernel name, template arguments, "
        "workgroup size and grid size (`grid threads`); `avg us (HIP events)` is what "
        "bench.py measured with events on the launch stream (including launch gaps).  "
        "The regimes run back to back in the timed steps; every other row is timed alone "
        "after a 1 GiB cache-evicting write.  The copy rows are the library's streaming "
        "copy (rowsm_stream_copy) of each regime's bytes with the same dtype pair; the "
        "fused copy row is a bf16 -> fp32 widening copy of as many elements as the causal "
        "mask keeps (the fused row's 1:2 read:write mix).  GB/s is algorithmic bytes "
        "over the rocprofv3 average.",
        "",
        "| row | workload | kernel | block | grid threads | calls | avg us (rocprofv3) | "
        "min us | max us | avg us (HIP events) | GB/s | % of peak |",
        "|---|---|---|---|---|---|---|---|---|---|---|---|",
    ]
    for (row, wl, spec, alg, ev_us, _key), got, shared in attribute(bench_targets(res), ds):
        if not got:
            lines.append(f"| {row} | {wl} | `{spec['base']}` | {spec['block']} | "
                         f"{spec['grid']} | 0 | - | - | - | - | - | - |")
            continue
        us = [d["us"] for d in got]
        avg = sum(us) / len(us)
        gbs = alg / (avg * 1e3)
        note = f" (shared with {', '.join(shared)})" if shared else ""
        ev = f"{ev_us:.2f}" if ev_us is not None else "-"
        lines.append(f"| {row} | {wl}{note} | `{_short(got[0]['name'])}` | {spec['block']} | "
                     f"{spec['grid']} | {len(us)} | {avg:.2f} | {min(us):.2f} | "
                     f"{max(us):.2f} | {ev} | {gbs:.0f} | {100 * gbs / peak_gbs:.1f} |")
    lines += ["", f"Whole-step value printed by that run: {res.get('value', 0):.0f} GB/s "
              f"({res.get('ms_per_step', 0):.3f} ms per step); peak {peak_gbs:.0f} GB/s.", "",
              "Algorithmic bytes: x read once plus y written once; for the fused row the "
              "kept entries of x; for the backward rows y and dy read once plus dx written "
              "once; for the MoE rows the scores read once plus the group scores written "
              "once."]
    return "\n".join(lines) + "\n"


def counter_values(rows: list, counter: str) -> list:
    """(dispatch, value) pairs of one counter from counter_collection rows."""
    per = {}
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        key = int(r.get("Dispatch_Id") or r.get("Correlation_Id") or 0)
        d = per.setdefault(key, {"row": r, "value": 0.0})
        d["value"] += float(r["Counter_Value"])
    out = []
    for key in sorted(per):
        r = per[key]["row"]
        base, args = parse_kernel_name(r.get("Kernel_Name", ""))
        out.append(({"name": r.get("Kernel_Name", ""), "base": base, "args": args,
                     "block": _size(r, "Workgroup_Size"), "grid": _size(r, "Grid_Size"),
                     "id": key}, per[key]["value"]))
    return out


def calibration_scale(cal_dir: str, counter: str, nbytes: int) -> float:
    """Bytes per counter KiB: a plain device copy of nbytes (the runtime's
    copyBuffer kernel) read through the same counter."""
    vals = [v for d, v in counter_values(read_csv_rows(cal_dir, "counter_collection.csv"),
                                         counter) if "copyBuffer" in d["name"]]
    if not vals:
        raise ValueError(f"no copyBuffer dispatch with {counter} in {cal_dir}")
    avg = sum(vals) / len(vals)
    return nbytes / (avg * 1024.0)


def summarize_counters(bench_log: str, fetch_dir: str, write_dir: str, cal_fetch_dir: str,
                       cal_write_dir: str, cal_bytes: int, commands: str, source_hash,
                       kernel_family):
    """(markdown, traffic table) from FETCH_SIZE and WRITE_SIZE runs of bench.py
    and of the calibration copy."""
    from paper_2607_23089_amd import workloads as W

    res = read_bench_json(bench_log)
    fs = calibration_scale(cal_fetch_dir, "FETCH_SIZE", cal_bytes)
    ws = calibration_scale(cal_write_dir, "WRITE_SIZE", cal_bytes)
    fetch = counter_values(read_csv_rows(fetch_dir, "counter_collection.csv"), "FETCH_SIZE")
    write = counter_values(read_csv_rows(write_dir, "counter_collection.csv"), "WRITE_SIZE")
    table = {"fetch_scale": fs, "write_scale": ws,
             "note": "per launch: kernel, launch shape, hash of the kernel family's device "
                     "sources", "launches": {}}
    lines = [
        "# HBM traffic counters: row-softmax regimes and the next rows", "",
        "Commands (repository root, MI355X; each counter in its own run):", "",
        "    " + commands.replace("\n", "\n    "), "",
        "Written by `python3 bench.py --summarize-counters`.  Calibration: a plain "
        f"{cal_bytes} B device copy (torch `copy_`, the runtime's copyBuffer kernel) gives "
        f"bytes = FETCH_SIZE x 1024 x {fs:.4f} and WRITE_SIZE x 1024 x {ws:.4f}.  Dispatches "
        "are matched to the launches of the bench JSON line by kernel name, template "
        "arguments, workgroup size and grid size.", "",
        "| row | workload | kernel | dispatches | input bytes | fetched bytes | fetch / input "
        "| output bytes | written bytes | write / output |",
        "|---|---|---|---|---|---|---|---|---|---|",
    ]
    targets = [t for t in bench_targets(res) if t[0] not in ("copy", "fused copy",
                                                             "launch_bound")]
    for row, wl, spec, alg, _ev, key in targets:
        fv = [v for d, v in fetch if matches(spec, d)]
        wv = [v for d, v in write if matches(spec, d)]
        if not fv or not wv:
            lines.append(f"| {row} | {wl} | `{spec['base']}` | 0 | | | | | | |")
            continue
        name = next(d["name"] for d, _v in fetch if matches(spec, d))
        fb = sum(fv) / len(fv) * 1024.0 * fs
        wb = sum(wv) / len(wv) * 1024.0 * ws
        inb, outb = io_bytes(row, wl, res, W)
        lines.append(f"| {row} | {wl} | `{_short(name)}` | {len(fv)} | {inb} | {fb:.4g} | "
                     f"{fb / inb:.4f} | {outb} | {wb:.4g} | {wb / outb:.4f} |")
        launch = launch_desc(row, wl, res)
        short = _short(name)
        table["launches"][key] = {
            "kernel": short, "launch": launch, "grid_threads": spec["grid"],
            "source_hash": source_hash(kernel_family(short)),
            "fetch_bytes": fb, "write_bytes": wb, "hbm_bytes_per_launch": fb + wb,
            "algorithmic_bytes": alg, "fetch_over_input_bytes": fb / inb,
            "write_over_output_bytes": wb / outb, "dispatches": len(fv)}
    lines += ["", "Input bytes: x (the kept entries of x for the fused row; y and dy for "
              "the backward rows; the scores for the MoE rows).  A ratio of 1.00 means every "
              "input byte is fetched once and every output byte written once."]
    return "\n".join(lines) + "\n", table


def launch_desc(row: str, wl: str, res: dict) -> str:
    if row == "regimes":
        return res["regimes_detail"][wl]["launch"]
    nxt = res["next_rows"]
    if row == "fused":
        return nxt["fused_scale_causal"]["launch"]
    return nxt[row][wl]["launch"]


def io_bytes(row: str, wl: str, res: dict, W) -> tuple:
    """(input bytes, output bytes) of one launch."""
    if row in ("regimes", "log_softmax"):
        w = W.WORKLOADS[wl]
        return w.rows * w.cols * w.in_bytes, w.rows * w.cols * w.out_bytes
    if row == "fused":
        w = W.WORKLOADS[wl]
        fz = res["next_rows"]["fused_scale_causal"]
        out = w.rows * w.cols * w.out_bytes
        return fz["algorithmic_bytes"] - out, out
    if row == "softmax_backward":
        w = W.BACKWARD_WORKLOADS[wl]
        return 2 * w.rows * w.cols * w.in_bytes, w.rows * w.cols * w.out_bytes
    w = W.MOE_WORKLOADS[wl]
    return (w.tokens * w.experts * w.in_bytes,
            w.tokens * (w.experts // w.group) * w.out_bytes)


def summarize_launcher(bench_log: str, trace_dir: str, command: str, peak_gbs: float) -> str:
    """The launcher check's kernel durations: the check's JSON line lists, per
    shape, the launch shapes it timed in order, each launched a fixed number of
    times (the last ones timed); dispatches of the library's row kernels are
    taken in that order."""
    res = read_bench_json(bench_log)
    per_shape = res["reps_per_shape"]
    untimed = 2
    ds = [d for d in dispatches(read_csv_rows(trace_dir, "kernel_trace.csv"))
          if d["base"] and d["base"] != "stream_copy_kernel"]
    need = sum(len(r["timed"]) for r in res["launcher_check"]) * per_shape
    if len(ds) != need:
        raise ValueError(f"{len(ds)} row-kernel dispatches in the trace, {need} expected")
    lines = [
        "# Launcher check: the launcher's choice against the library's other launch shapes "
        "(kernel trace)", "",
        "Command (repository root, MI355X):", "",
        "    " + command.replace("\n", "\n    "), "",
        "Written by `python3 bench.py --summarize-launcher`.  For launches of representative "
        "row lengths and counts, bench.py --launcher-check times the launcher's choice "
        "(`auto`) and every other launch shape of the library that takes the shape: medium "
        "groups of w waves with the default rows per block (`Mw`) or one row per block "
        "(`Mwr1`), the single-read form with S blocks of T threads per row (`SsTt`), and "
        "for rows of at most 256 columns the grid capped at N = 4-128 blocks per compute "
        "unit (`bpcN`) and blocks of b threads with r row groups per lane (`bBrR`); each "
        "launch alone after a "
        f"1 GiB cache-evicting write, {untimed} untimed and {per_shape - untimed} timed "
        "launches per shape.  Times are the rocprofv3 durations of the timed launches, "
        "matched to their shape in launch order.", "",
        "| op | rows x cols | dtypes | launcher's choice | auto us | best shape | best us | "
        "auto / best | auto GB/s | % of peak |",
        "|---|---|---|---|---|---|---|---|---|---|",
    ]
    i = 0
    ratios = []
    for r in res["launcher_check"]:
        us = {}
        for name in r["timed"]:
            got = ds[i:i + per_shape]
            i += per_shape
            if name == "auto":
                op = {"scaled_causal": "scaled_causal", "backward": "backward"}.get(
                    r["op"], "softmax")
                spec = launch_spec(op, r["launch"], r["in"], r["out"])
                if not all(matches(spec, d) for d in got):
                    raise ValueError(f"dispatches of {r['op']} {r['rows']}x{r['cols']} auto "
                                     f"do not match {r['launch']}")
            t = [d["us"] for d in got[untimed:]]
            us[name] = sum(t) / len(t)
        best = min(us, key=us.get)
        ib, ob = DTYPE_BYTES[r["in"]], DTYPE_BYTES[r["out"]]
        n = r["rows"] * r["cols"]
        if r["op"] == "backward":
            alg = n * (2 * ib + ob)
        elif r["op"] == "scaled_causal":
            # the kept entries of x (column c of row r kept for c <= r mod q,
            # q = causal_period; the launcher check passes q = cols) and all of y
            q = r.get("causal_period") or r["cols"]
            full, rem = divmod(r["rows"], q)
            kept = full * (q * (q + 1) // 2) + rem * (rem + 1) // 2
            alg = kept * ib + n * ob
        else:
            alg = n * (ib + ob)
        gbs = alg / (us["auto"] * 1e3)
        f = parse_launch(r["launch"])
        choice = (f"{f['family']} wpr={f.get('wpr')} nv={f.get('nv')} split={f.get('split')} "
                  f"block={f.get('block')}")
        lines.append(f"| {r['op']} | {r['rows']} x {r['cols']} | {r['in']} -> {r['out']} | "
                     f"{choice} | {us['auto']:.1f} | {best} | {us[best]:.1f} | "
                     f"{us['auto'] / us[best]:.3f} | {gbs:.0f} | {100 * gbs / peak_gbs:.1f} |")
        ratios.append(us["auto"] / us[best])
    gm = 1.0
    for q in ratios:
        gm *= q ** (1.0 / len(ratios))
    lines += ["", f"The launcher's choice over the fastest shape: geometric mean {gm:.3f} over "
              f"{len(ratios)} launches, at most {max(ratios):.3f}.  Algorithmic bytes: x read "
              "once and y written once (the kept entries of x for the fused rows; y and dy "
              "for the backward)."]
    return "\n".join(lines) + "\n"


def summarize_sweep(bench_log: str, trace_dir: str, command: str, peak_gbs: float) -> str:
    """Size sweep: per size, the kernel's and the copy's rocprofv3 durations
    (timed launches, in launch order), and a least-squares line
    duration = t0 + bytes / rate over the sizes of at least 64 MiB."""
    res = read_bench_json(bench_log)
    per = res["launches_per_size"]
    untimed = 2
    ds = [d for d in dispatches(read_csv_rows(trace_dir, "kernel_trace.csv"))
          if d["base"] in ("small_row_kernel", "medium_row_kernel", "stream_copy_kernel")]
    need = 2 * per * len(res["size_sweep"])
    if len(ds) != need:
        raise ValueError(f"{len(ds)} dispatches in the trace, {need} expected")
    rows, pts = [], []
    i = 0
    for s in res["size_sweep"]:
        k, c = ds[i:i + per], ds[i + per:i + 2 * per]
        i += 2 * per
        spec = launch_spec("softmax", s["launch"], "bf16", "bf16")
        if not all(matches(spec, d) for d in k) or any(d["base"] != "stream_copy_kernel"
                                                        for d in c):
            raise ValueError(f"dispatches of {s['rows']} rows do not match {s['launch']}")
        kt = sorted(d["us"] for d in k[untimed:])
        ct = sorted(d["us"] for d in c[untimed:])
        km, cm = kt[len(kt) // 2], ct[len(ct) // 2]
        rows.append((s, km, cm, _short(k[0]["name"]), k[0]["block"], k[0]["grid"]))
        if s["bytes"] >= 64 << 20:
            pts.append((s["bytes"], km))
    n = len(pts)
    mb = sum(b for b, _ in pts) / n
    mt = sum(t for _, t in pts) / n
    slope = sum((b - mb) * (t - mt) for b, t in pts) / sum((b - mb) ** 2 for b, _ in pts)
    t0 = mt - slope * mb
    rate = 1.0 / slope / 1e3  # GB/s (bytes per us / 1e3)
    lines = [
        "# Size sweep: small-row kernel and plain copy from 4 MiB to 1 GiB (kernel trace)", "",
        "Command (repository root, MI355X):", "",
        "    " + command.replace("\n", "\n    "), "",
        "Written by `python3 bench.py --summarize-sweep`.  The small-row workload's shape "
        "(64 bf16 columns, bf16 output) at 16384 to 4194304 rows, the launcher's choice at "
        "each, and the library's streaming copy of the same bytes; each launch alone after a "
        f"1 GiB cache-evicting write, {untimed} untimed and {per - untimed} timed launches "
        "each; medians of the timed launches' rocprofv3 durations.  Bytes: x read plus y "
        "written.", "",
        "| rows | MiB | kernel | block | grid threads | kernel us | GB/s | % of peak | copy us "
        "| copy GB/s |",
        "|---|---|---|---|---|---|---|---|---|---|",
    ]
    for s, km, cm, name, blk, grid in rows:
        g = s["bytes"] / (km * 1e3)
        lines.append(f"| {s['rows']} | {s['bytes'] >> 20} | `{name}` | {blk} | {grid} | "
                     f"{km:.2f} | {g:.0f} | {100 * g / peak_gbs:.1f} | {cm:.2f} | "
                     f"{s['bytes'] / (cm * 1e3):.0f} |")
    lines += ["", f"Least-squares line over the {n} sizes of at least 64 MiB: duration = "
              f"{t0:.2f} us + bytes / {rate:.0f} GB/s ({100 * rate / peak_gbs:.1f}% of peak)."]
    return "\n".join(lines) + "\n"


def summarize_pmc(bench_log: str, pmc_dir: str, command: str) -> str:
    """Per-launch averages of every counter in a rocprofv3 --pmc run of bench.py."""
    res = read_bench_json(bench_log)
    rows = read_csv_rows(pmc_dir, "counter_collection.csv")
    names = sorted({r["Counter_Name"] for r in rows})
    vals = {n: counter_values(rows, n) for n in names}
    lines = [
        "# Counters per launch: " + ", ".join(names), "",
        "Command (repository root, MI355X):", "",
        "    " + command.replace("\n", "\n    "), "",
        "Written by `python3 bench.py --summarize-pmc`: the average of each counter over the "
        "dispatches of each launch of the bench JSON line, matched by kernel name, template "
        "arguments, workgroup size and grid size.", "",
        "| row | workload | kernel | dispatches | " + " | ".join(names) + " |",
        "|---|---|---|---|" + "---|" * len(names),
    ]
    for row, wl, spec, _alg, _ev, _key in bench_targets(res):
        per = [[v for d, v in vals[n] if matches(spec, d)] for n in names]
        if not per[0]:
            continue
        name = next(d["name"] for d, _v in vals[names[0]] if matches(spec, d))
        cells = " | ".join(f"{sum(v) / len(v):.4g}" if v else "-" for v in per)
        lines.append(f"| {row} | {wl} | `{_short(name)}` | {len(per[0])} | {cells} |")
    return "\n".join(lines) + "\n"


def summarize_overlap(bench_log: str, trace_dir: str, command: str) -> str:
    """Overlap in time of the two streams' dispatches of bench.py
    --stream-overlap: the dispatches of launch A and of launch B after the
    reference and warm-up launches, paired in issue order.  (Their grid is
    sized from occupancy at launch, so they are matched by kernel, template
    arguments and workgroup size.)"""
    res = read_bench_json(bench_log)["stream_overlap"]
    ds = [d for d in dispatches(read_csv_rows(trace_dir, "kernel_trace.csv"))
          if d["base"] in ("split_row_kernel", "large_row_kernel")]
    sa = dict(launch_spec("softmax", res["launch_a"], "f32", "f32"), grid=None)
    sb = dict(launch_spec("softmax", res["launch_b"], "bf16", "f32"), grid=None)

    def like(spec, d):
        return matches(dict(spec, grid=d["grid"]), d)

    skip = 1 + res.get("warm_up_launches", 0) // 2
    a = [d for d in ds if like(sa, d)][skip:]
    b = [d for d in ds if like(sb, d)][skip:]
    n = res["pairs"]
    if len(a) != n or len(b) != n:
        raise ValueError(f"{len(a)} and {len(b)} dispatches, {n} pairs expected")
    lines = [
        "# Two unordered streams: overlap in time of exchanging launches (kernel trace)", "",
        "Command (repository root, MI355X):", "",
        "    " + command.replace("\n", "\n    "), "",
        "Written by `python3 bench.py --summarize-overlap`.  bench.py --stream-overlap issues "
        f"{n} pairs of launches, A on one stream and B on another, never ordered against "
        "each other (after one launch on each stream, so that neither stream's first use "
        "falls inside the pairs).  Both take the single-read form, whose blocks exchange "
        "their partial results through the library's exchange ring, capped at one block "
        "per compute unit so that each leaves room for the other.  Every output equals the "
        "same launch made alone, bitwise (`outputs_equal_to_launches_alone`: "
        f"{res['outputs_equal_to_launches_alone']}).", "",
        f"- A: {res.get('rows_a', '?')} x 262144 f32 -> f32, `{res['launch_a']}`",
        f"- B: {res.get('rows_b', '?')} x 151936 bf16 -> f32, `{res['launch_b']}`", "",
        "| launch | stream | start (us) | end (us) | us | time shared with the other stream's "
        "kernels (us) |",
        "|---|---|---|---|---|---|",
    ]
    iv = lambda d: (int(d["row"]["Start_Timestamp"]), int(d["row"]["End_Timestamp"]))
    ia, ib = [iv(d) for d in a], [iv(d) for d in b]
    t0 = min(ia[0][0], ib[0][0])
    shared = lambda x, others: sum(max(0, min(x[1], o[1]) - max(x[0], o[0])) for o in others)
    rows = sorted([("A", i, x, shared(x, ib)) for i, x in enumerate(ia)] +
                  [("B", i, x, shared(x, ia)) for i, x in enumerate(ib)], key=lambda r: r[2][0])
    for lab, i, (x0, x1), sh in rows:
        lines.append(f"| {lab}{i} | {lab} | {(x0 - t0) / 1e3:.1f} | {(x1 - t0) / 1e3:.1f} | "
                     f"{(x1 - x0) / 1e3:.1f} | {sh / 1e3:.1f} |")
    both = sum(shared(x, ib) for x in ia)
    span = max(ia[-1][1], ib[-1][1]) - t0
    lines += ["", f"Both streams had a kernel running for {both / 1e3:.1f} us of the "
              f"{span / 1e3:.1f} us from the first pair's first start to the last end "
              f"({100 * both / span:.0f}%); {sum(1 for _l, _i, _x, sh in rows if sh > 0)} of "
              f"{len(rows)} launches ran partly alongside the other stream's."]
    return "\n".join(lines) + "\n"
