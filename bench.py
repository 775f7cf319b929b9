#!/usr/bin/env python3
"""Row-softmax benchmark on one MI355X.

One step is one pass of the whole hot path over one batch of each row-length
regime, in this order (inputs resident in HBM before timing starts):

  small_262144x64    bf16 -> bf16   small-row kernel
  causal_32768x4096  bf16 -> bf16   medium-row kernel
  large_1024x262144  f32  -> f32    large-row kernel
  vocab_4096x151936  bf16 -> f32    launcher's choice for 151936-wide rows

Between two visits of the same input the other three move more than 3 GB, far
more than the 256 MB memory-side cache plus L2, so every launch reads x from
HBM.  ``value`` is the step's algorithmic bytes (x read once + y written
once, summed over the regimes) divided by the step time: the host clock over
K back-to-back steps between two device synchronisations.  Per-launch times
come from a separate pass of K steps in which each launch is bracketed by
HIP timing events (created without a system-scope fence) recorded on the
stream it runs on.

The same four launches are also captured into one HIP graph and replayed
(``graph_step``).

Before the timed steps the same protocol times the library's streaming copy
(rowsm_stream_copy) of each regime's bytes, same dtype pair and buffers: a
plain copy moving the same bytes in the same run, reported per launch as
``ratio_to_copy`` (kernel rate / copy rate).

Parity gate: before anything is timed, one untimed step runs and its outputs
are checked against the fp64 oracle on sampled rows of every regime (first and
last rows and evenly spaced ones); a failure prints a line with no value and
exits non-zero.  After timing, the CPU baseline checks every 16th row of the
timed steps' outputs on the way, with the same consequence on failure.

Prints ONE JSON line (rank 0).  ``--gpus`` above 1 is refused: this path runs
on one GPU (rows shard across GPUs without communication).

``--summarize-trace``, ``--summarize-counters`` and ``--summarize-launcher``
need no GPU: they write the summaries under profiles/ from the CSV output of
rocprofv3 runs of this script (bench_profiles.py).

``--launcher-check`` runs no step: it times the launcher's choice for full
launches of representative row lengths against the library's other launch
shapes (each launch alone after a cache-evicting write) and prints that as
the JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "row-softmax achieved HBM GB/s and % of MI355X peak, per row-length regime"
PEAK_HBM_GBS = 8000.0  # MI355X published HBM3E bandwidth
# Bandwidth targets per regime, as fractions of the HBM peak: at least 60%
# for the small-row regime, 80% for medium and long rows.
TARGET_FRAC = {"small_262144x64": 0.60, "causal_32768x4096": 0.80,
               "large_1024x262144": 0.80, "vocab_4096x151936": 0.80}
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "hbm_traffic.json")
# hipDeviceAttribute_t values of the HIP runtime headers (hip_runtime_api.h).
HIP_ATTR_MEMORY_BUS_WIDTH = 59
HIP_ATTR_MEMORY_CLOCK_RATE = 60
# Device code each kernel family is compiled from; a profile entry records the
# hash of its family's sources and the launch's shape.
KERNEL_SOURCES = {
    "small_row": ["rowsm_device.hpp", "small_row.hpp"],
    "medium_row": ["rowsm_device.hpp", "medium_row.hpp"],
    "split_row": ["rowsm_device.hpp", "split_row.hpp"],
    "large_row": ["rowsm_device.hpp", "large_row.hpp"],
    "bwd": ["rowsm_device.hpp", "medium_row.hpp", "split_row.hpp", "backward_row.hpp"],
    "group_top2": ["rowsm_device.hpp", "group_top2.hpp"],
}


def kernel_family(kernel: str) -> str:
    """Family of a kernel name (e.g. 'split_row_kernel<...>' -> 'split_row')."""
    if kernel.startswith("bwd_"):
        return "bwd"
    return kernel.split("_kernel")[0]


def kernel_source_hash(family: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[family]:
        with open(os.path.join(ROOT, "paper_2607_23089_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(key: str, launch: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when there is none, or the device code of that launch's kernel
    family or the launch's shape changed since it was taken."""
    try:
        with open(PROFILE_COUNTERS) as f:
            prof = json.load(f)
    except (OSError, ValueError):
        return None
    ent = prof.get("launches", {}).get(key)
    if ent is None or ent.get("launch") != launch:
        return None
    fam = kernel_family(ent.get("kernel", ""))
    if fam not in KERNEL_SOURCES or ent.get("source_hash") != kernel_source_hash(fam):
        return None
    return ent.get("hbm_bytes_per_launch")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def copy_ceiling(reps: int = 10):
    """Same-run context: torch's device copy (the runtime's copy kernel) and
    fill of 1 GiB, timed like the next-row legs."""
    import torch
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    a = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    copy_us = timed_alone(lambda: b.copy_(a), reps, flush, stream)
    fill_us = timed_alone(lambda: b.zero_(), reps, flush, stream)
    nbytes = a.numel() * 4
    props = torch.cuda.get_device_properties(dev)
    return {"torch_copy_1GiB_GBps": 2 * nbytes / (copy_us * 1e3),
            "torch_fill_1GiB_GBps": nbytes / (fill_us * 1e3),
            "read_write_model_read_GBps": MEASURED_READ_GBS,
            "read_write_model_write_GBps": MEASURED_WRITE_GBS,
            "device": props.name, "gcn_arch": getattr(props, "gcnArchName", None),
            "compute_units": props.multi_processor_count}


def cpu_baseline(inputs, outputs, regimes, min_seconds: float, threads: int = 0):
    """Time the fp64 oracle on the host cores over every row of the step (row
    chunks bounded in memory), repeating passes until ``min_seconds`` of
    oracle time has accumulated, and check evenly spaced GPU rows against it
    on the way."""
    import numpy as np

    import oracle
    from oracle.compare import compare, widen_output
    from paper_2607_23089_amd import workloads as W

    threads = threads or len(os.sched_getaffinity(0))
    oracle.load()
    chunk_elems = 1 << 25
    tot_bytes, tot_time, passes = 0, 0.0, 0
    parity = {}
    widened = {}  # host fp64 copies of the inputs, kept for repeated passes
    while passes == 0 or tot_time < min_seconds:
        for name in regimes:
            w = W.WORKLOADS[name]
            step_rows = max(1, chunk_elems // w.cols)
            for r0 in range(0, w.rows, step_rows):
                v = widened.get((name, r0))
                if v is None:
                    xs = W.to_bits_numpy(inputs[name][r0:r0 + step_rows])
                    v = (oracle.widen_bf16_bits(xs) if w.in_dtype == "bf16"
                         else oracle.widen_f32(xs))
                    widened[(name, r0)] = v
                t = time.perf_counter()
                ref = oracle.softmax_f64(v, threads=threads)
                tot_time += time.perf_counter() - t
                tot_bytes += v.size * (w.in_bytes + w.out_bytes)
                if passes == 0:
                    # parity on every 16th row of the chunk
                    got = widen_output(W.to_bits_numpy(outputs[name][r0:r0 + step_rows:16]),
                                       w.out_dtype)
                    res = compare(got, ref[::16], w.out_dtype)
                    p = parity.setdefault(name, {"rows_checked": 0, "parity_ok": True,
                                                 "max_abs": 0.0, "max_rel": 0.0,
                                                 "max_tol_ratio": 0.0})
                    p["rows_checked"] += int(got.shape[0])
                    p["parity_ok"] &= bool(res["ok"])
                    p["max_abs"] = max(p["max_abs"], res["max_abs"])
                    # relative error over entries of magnitude >= 1e-30 (reported,
                    # not gated: the fp32 bound is absolute)
                    p["max_rel"] = max(p["max_rel"], res["max_rel"])
                    p["max_tol_ratio"] = max(p["max_tol_ratio"], res["max_tol_ratio"])
        passes += 1
    # one thread on one chunk of the longest-row regime, for scale
    name = max(regimes, key=lambda n: W.WORKLOADS[n].cols)
    v1 = widened[(name, 0)]
    t = time.perf_counter()
    oracle.softmax_f64(v1, threads=1)
    t1 = time.perf_counter() - t
    w1 = W.WORKLOADS[name]
    return {
        "value": tot_bytes / tot_time / 1e9,
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"every row of the step ({', '.join(regimes)}), {passes} pass(es), "
                   f"{tot_time:.1f} s of oracle time; widening and copies not timed"),
        "seconds": tot_time,
        "single_thread_GBps": v1.size * (w1.in_bytes + w1.out_bytes) / t1 / 1e9,
        "single_thread_sample": f"{v1.shape[0]} rows of {name}",
        "cpu_model": cpu_model(),
        "parity_on_sample": parity,
    }


def gate_rows(rows: int, n: int = 24):
    """Rows the parity gate checks: the first and last four and n evenly spaced
    ones in between (row 0 and every 4096th row are the causal workload's
    one-hot rows)."""
    picks = set(range(min(4, rows))) | set(range(max(0, rows - 4), rows))
    picks |= {(i * (rows - 1)) // max(1, n - 1) for i in range(n)}
    return sorted(picks)


def parity_gate(inputs, outputs, regimes, threads: int = 0):
    """Parity of the launches the bench times, checked before any timing: the
    outputs of one untimed step against the fp64 oracle on sampled rows of
    every regime (compare(): NaN and zero patterns exact, 2e-6 absolute for
    fp32 output, one bf16 ulp of the oracle value for bf16 output)."""
    import torch

    import oracle
    from oracle.compare import compare, widen_output
    from paper_2607_23089_amd import workloads as W

    threads = threads or len(os.sched_getaffinity(0))
    oracle.load()
    out = {}
    for name in regimes:
        w = W.WORKLOADS[name]
        rows = gate_rows(w.rows)
        ti = torch.tensor(rows, dtype=torch.int64, device=inputs[name].device)
        xs = W.to_bits_numpy(inputs[name].index_select(0, ti))
        v = oracle.widen_bf16_bits(xs) if w.in_dtype == "bf16" else oracle.widen_f32(xs)
        ref = oracle.softmax_f64(v, threads=threads)
        got = widen_output(W.to_bits_numpy(outputs[name].index_select(0, ti)), w.out_dtype)
        res = compare(got, ref, w.out_dtype)
        out[name] = {"rows_checked": len(rows), "parity_ok": bool(res["ok"]),
                     "max_abs": res["max_abs"], "max_tol_ratio": res["max_tol_ratio"]}
    return out


def device_memory_info(device_index: int = 0):
    """The device-reported HBM figures (hipDeviceGetAttribute): memory clock
    in kHz and bus width in bits."""
    import ctypes
    h = ctypes.CDLL("libamdhip64.so")
    h.hipDeviceGetAttribute.argtypes = [ctypes.POINTER(ctypes.c_int), ctypes.c_int, ctypes.c_int]
    vals = {}
    for key, attr in (("memory_clock_khz", HIP_ATTR_MEMORY_CLOCK_RATE),
                      ("bus_width_bits", HIP_ATTR_MEMORY_BUS_WIDTH)):
        v = ctypes.c_int(0)
        st = h.hipDeviceGetAttribute(ctypes.byref(v), attr, device_index)
        vals[key] = v.value if st == 0 else None
    return vals


class HipEvent:
    """A HIP timing event created without a system-scope fence (HIP's
    hipEventDisableSystemFence), recorded on the stream the kernel runs on.
    Timing events need no fence; torch's events carry one, which added about
    8 us to each 4-launch step and 1.7 us to a 13 us launch."""
    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        import ctypes
        if HipEvent._hip is None:
            h = ctypes.CDLL("libamdhip64.so")
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                              ctypes.c_void_p]
            h.hipEventDestroy.argtypes = [ctypes.c_void_p]
            HipEvent._hip = h
        self._ct = ctypes
        self.ev = ctypes.c_void_p()
        if HipEvent._hip.hipEventCreateWithFlags(ctypes.byref(self.ev),
                                                 self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream):
        if HipEvent._hip.hipEventRecord(self.ev, self._ct.c_void_p(stream.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end) -> float:
        """Milliseconds from this event to ``end`` (both complete)."""
        ms = self._ct.c_float()
        if HipEvent._hip.hipEventElapsedTime(self._ct.byref(ms), self.ev, end.ev) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        # through type(self): at interpreter exit the module's globals may
        # already be cleared when a module-level event is collected
        hip = type(self)._hip
        if hip is not None and self.ev:
            hip.hipEventDestroy(self.ev)


# Read-only and write-only rates of streaming probes with 8 vectors per
# thread, an early model of a read/write mix: 1 / (r / READ + (1 - r) / WRITE)
# for read fraction r.  It is a model, not a bound (streams with one vector
# per thread, the long-row kernels among them, exceed it); the same-run copy
# of the same byte mix (ratio_to_copy) is the reference where one exists.
MEASURED_READ_GBS = 6870.0
MEASURED_WRITE_GBS = 5950.0


def mix_bound_gbs(read_bytes: float, write_bytes: float) -> float:
    tot = read_bytes + write_bytes
    return tot / (read_bytes / MEASURED_READ_GBS + write_bytes / MEASURED_WRITE_GBS)


def timed_alone(fn, reps: int, flush, stream) -> float:
    """Average microseconds of fn() over reps launches (after 2 untimed),
    each preceded by a 1 GiB write that evicts the memory-side cache."""
    import torch
    ts = []
    for i in range(reps + 2):
        flush.zero_()
        e0, e1 = HipEvent(), HipEvent()
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        if i >= 2:
            ts.append(e0.elapsed_time(e1))
    return sum(ts) / len(ts) * 1e3


def log_softmax_leg(reps: int):
    """Log-softmax on the long-row workloads (its cross-entropy use), each
    launch timed alone, next to softmax on the same input under the same
    protocol, and the library's streaming copy of the same bytes (same dtype
    pair and buffers).  Algorithmic bytes: x read once plus y written once."""
    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    out = {}
    for name in ("vocab_4096x151936", "large_1024x262144"):
        w = W.WORKLOADS[name]
        x = W.make_input(w, device=dev)
        y = torch.empty(w.rows, w.cols, dtype=W.TORCH_DTYPES[w.out_dtype], device=dev)
        di, do = R.dtype_code(x.dtype), R.dtype_code(y.dtype)
        log_us = timed_alone(lambda: R.check(R.rowsm_log_softmax(
            x.data_ptr(), y.data_ptr(), w.rows, w.cols, di, do, sh, None)), reps, flush, stream)
        sm_us = timed_alone(lambda: R.check(R.rowsm_forward(
            x.data_ptr(), y.data_ptr(), w.rows, w.cols, di, do, sh)), reps, flush, stream)
        copy_us = timed_alone(lambda: R.check(R.rowsm_stream_copy(
            x.data_ptr(), y.data_ptr(), w.rows * w.cols, di, do, sh)), reps, flush, stream)
        gbs = w.algorithmic_bytes / (log_us * 1e-6) / 1e9
        copy_gbs = w.algorithmic_bytes / (copy_us * 1e-6) / 1e9
        bound = mix_bound_gbs(w.rows * w.cols * w.in_bytes, w.rows * w.cols * w.out_bytes)
        _, desc = R.rowsm_describe_op(R.OP_LOG_SOFTMAX, w.rows, w.cols, di, do)
        out[name] = {
            "launch": desc, "hbm_bytes_per_launch": measured_traffic(f"log_softmax/{name}", desc),
            "algorithmic_bytes": w.algorithmic_bytes, "avg_us": log_us,
            "GBps": gbs, "frac_of_peak": gbs / PEAK_HBM_GBS,
            "frac_of_read_write_model": gbs / bound,
            "softmax_same_protocol_us": sm_us,
            "copy_us": copy_us, "copy_GBps": copy_gbs, "ratio_to_copy": gbs / copy_gbs,
        }
        del x, y
    return out


def backward_leg(reps: int):
    """Softmax backward on the backward workloads, each launch timed alone.
    Algorithmic bytes: y and dy read once plus dx written once."""
    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    out = {}
    for name, w in W.BACKWARD_WORKLOADS.items():
        y, dy = W.make_backward_inputs(w, device=dev)
        dx = torch.empty(w.rows, w.cols, dtype=W.TORCH_DTYPES[w.out_dtype], device=dev)
        di, do = R.dtype_code(y.dtype), R.dtype_code(dx.dtype)
        us = timed_alone(lambda: R.check(R.rowsm_softmax_backward(
            y.data_ptr(), dy.data_ptr(), dx.data_ptr(), w.rows, w.cols, di, do, sh)),
            reps, flush, stream)
        gbs = w.algorithmic_bytes / (us * 1e-6) / 1e9
        bound = mix_bound_gbs(2 * w.rows * w.cols * w.in_bytes, w.rows * w.cols * w.out_bytes)
        _, desc = R.rowsm_describe_op(R.OP_SOFTMAX_BACKWARD, w.rows, w.cols, di, do)
        out[name] = {
            "launch": desc, "hbm_bytes_per_launch": measured_traffic(f"softmax_backward/{name}", desc),
            "algorithmic_bytes": w.algorithmic_bytes, "avg_us": us,
            "GBps": gbs, "frac_of_peak": gbs / PEAK_HBM_GBS,
            "frac_of_read_write_model": gbs / bound,
        }
        del y, dy, dx
    if R.rowsm_split_wait_failures() != 0:
        raise R.RowsmError("split-row exchange waits gave up: results invalid")
    return out


def moe_leg(reps: int):
    """MoE group score (sum of the two largest of each group of 32 expert
    scores) on the MoE workloads, each launch timed alone.  Algorithmic
    bytes: scores read once plus group scores written once."""
    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    out = {}
    for name, w in W.MOE_WORKLOADS.items():
        x = W.make_moe_scores(w, device=dev)
        o = torch.empty(w.tokens, w.experts // w.group, dtype=W.TORCH_DTYPES[w.out_dtype],
                        device=dev)
        di, do = R.dtype_code(x.dtype), R.dtype_code(o.dtype)
        us = timed_alone(lambda: R.check(R.rowsm_moe_group_top2(
            x.data_ptr(), o.data_ptr(), w.tokens, w.experts, w.group, di, do, sh)),
            reps, flush, stream)
        gbs = w.algorithmic_bytes / (us * 1e-6) / 1e9
        n = w.tokens * w.experts
        bound = mix_bound_gbs(n * w.in_bytes, n // w.group * w.out_bytes)
        _, desc = R.rowsm_describe_op(R.OP_MOE_GROUP_TOP2, n // w.group, w.group, di, do)
        out[name] = {
            "launch": desc, "hbm_bytes_per_launch": measured_traffic(f"moe_group_top2/{name}", desc),
            "algorithmic_bytes": w.algorithmic_bytes, "avg_us": us,
            "GBps": gbs, "frac_of_peak": gbs / PEAK_HBM_GBS,
            "frac_of_read_write_model": gbs / bound,
        }
        del x, o
    return out


def launch_bound_leg(reps: int):
    """The 64 x 1000 fp32 workload, 256 KB: launch bound, so timed two ways,
    each launch alone between events, and many launches back to back between
    one event pair (the per-launch cost of a stream of such launches)."""
    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    w = W.WORKLOADS["fp32_64x1000"]
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    x = W.make_input(w, device=dev)
    y = torch.empty_like(x)

    def launch():
        R.check(R.rowsm_forward(x.data_ptr(), y.data_ptr(), w.rows, w.cols, R.F32, R.F32, sh))

    for _ in range(10):
        launch()
    torch.cuda.synchronize()
    alone = []
    for _ in range(reps):
        e0, e1 = HipEvent(), HipEvent()
        e0.record(stream)
        launch()
        e1.record(stream)
        torch.cuda.synchronize()
        alone.append(e0.elapsed_time(e1) * 1e3)
    alone.sort()
    n = 200
    e0, e1 = HipEvent(), HipEvent()
    e0.record(stream)
    for _ in range(n):
        launch()
    e1.record(stream)
    torch.cuda.synchronize()
    _, desc = R.rowsm_describe(w.rows, w.cols, R.F32, R.F32)
    return {"workload": "fp32_64x1000 f32->f32 (parity workload; 256 KB, launch bound)",
            "launch": desc, "median_us_alone": alone[len(alone) // 2],
            "us_per_launch_back_to_back": e0.elapsed_time(e1) * 1e3 / n}


def fused_causal_leg(reps: int):
    """The fused form (scale and causal mask computed in the kernel) on the
    causal workload's shape, next to the plain form on the same scores with
    the mask stored as -inf.  Each launch is timed alone after a 1 GiB write
    that evicts the memory-side cache.  Algorithmic bytes of the fused form:
    the kept entries of x read once plus all of y written once.  A widening
    streaming copy with the same read:write mix is timed beside it."""
    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    w = W.WORKLOADS["causal_32768x4096"]
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(0)
    x = (torch.randn(w.rows, w.cols, generator=g, device=dev) * w.sigma).to(torch.bfloat16)
    xm = W.make_input(w, device=dev)
    y = torch.empty_like(x)
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    scale = 0.125  # 1/sqrt(64), a head dimension of 64

    def timed(fn):
        return timed_alone(fn, reps, flush, stream)

    sh = stream.cuda_stream
    fused_us = timed(lambda: R.check(R.rowsm_forward_scaled_causal(
        x.data_ptr(), y.data_ptr(), w.rows, w.cols, R.BF16, R.BF16, scale, w.period, 0, sh)))
    plain_us = timed(lambda: R.check(R.rowsm_forward(
        xm.data_ptr(), y.data_ptr(), w.rows, w.cols, R.BF16, R.BF16, sh)))
    q = w.period
    kept = (w.rows // q) * (q * (q + 1) // 2)
    alg = kept * w.in_bytes + w.rows * w.cols * w.out_bytes
    gbs = alg / (fused_us * 1e-6) / 1e9
    # The same 1:2 read:write mix as a plain stream: a bf16 -> fp32 widening
    # copy of `kept` elements reads the kept bytes and writes twice as many.
    wide = torch.empty(kept, dtype=torch.float32, device=dev)
    copy_us = timed(lambda: R.check(R.rowsm_stream_copy(
        x.data_ptr(), wide.data_ptr(), kept, R.BF16, R.F32, sh)))
    copy_gbs = kept * 6 / (copy_us * 1e-6) / 1e9
    del wide
    _, desc = R.rowsm_describe_op(R.OP_SCALED_CAUSAL, w.rows, w.cols, R.BF16, R.BF16)
    return {
        "workload": "causal_32768x4096 scores without stored mask, scale 0.125, "
                    "mask (r, c) = -inf for c > r mod 4096 computed in the kernel",
        "launch": desc, "copy_elements": kept,
        "algorithmic_bytes": alg, "kept_fraction": kept / (w.rows * w.cols),
        "avg_us": fused_us, "GBps": gbs, "frac_of_peak": gbs / PEAK_HBM_GBS,
        "stored_mask_same_protocol_us": plain_us, "speedup_vs_stored_mask": plain_us / fused_us,
        "copy_1to2_us": copy_us, "copy_1to2_GBps": copy_gbs, "ratio_to_copy": gbs / copy_gbs,
    }


LAUNCHER_SHAPES = [  # (op, rows, cols, in dtype, out dtype)
    ("softmax", 262144, 64, "bf16", "bf16"),
    ("softmax", 4194304, 64, "bf16", "bf16"),
    ("softmax", 32768, 4096, "f32", "f32"),
    ("softmax", 65536, 2048, "bf16", "f32"),
    ("softmax", 20480, 9216, "bf16", "bf16"),
    ("softmax", 16384, 8192, "f32", "f32"),
    ("softmax", 20480, 12288, "bf16", "bf16"),
    ("softmax", 20480, 10240, "bf16", "f32"),
    ("softmax", 2048, 12288, "bf16", "bf16"),
    ("softmax", 1024, 8192, "f32", "f32"),
    ("scaled_causal", 16384, 4096, "f32", "f32"),
    ("scaled_causal", 32768, 16384, "f32", "f32"),
    ("backward", 1024, 8192, "f32", "f32"),
    ("backward", 32768, 4096, "bf16", "bf16"),
    ("backward", 524288, 128, "bf16", "bf16"),
    ("backward", 131072, 64, "bf16", "bf16"),
    ("softmax", 1000003, 37, "f32", "f32"),      # one-wave rows, looping grid
    ("softmax", 1048576, 21, "bf16", "bf16"),    # small rows of one-element vectors
    ("softmax", 12288, 4001, "bf16", "bf16"),    # ragged width
    ("backward", 204600, 41, "bf16", "bf16"),    # one-wave rows, looping grid
]


SWEEP_ROWS = (16384, 32768, 65536, 131072, 262144, 524288, 1048576, 2097152, 4194304)


def size_sweep(reps: int = 10):
    """The small-row workload's kernel at 4 MiB to 1 GiB (64 bf16 columns, the
    launcher's choice at each row count), next to the library's streaming copy
    of the same bytes; every launch alone after a 1 GiB cache-evicting write,
    2 untimed and reps timed launches each, kernel before copy, sizes in
    order.  A kernel trace of this run gives duration against bytes: the
    fixed cost of a launch and the rate it approaches."""
    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    sh = stream.cuda_stream
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    out = []
    for rows in SWEEP_ROWS:
        x = W.random_matrix(rows, 64, "bf16", sigma=4.0, seed=1, device=dev)
        y = torch.empty_like(x)
        kern = timed_alone(lambda: R.check(R.rowsm_forward(
            x.data_ptr(), y.data_ptr(), rows, 64, R.BF16, R.BF16, sh)), reps, flush, stream)
        copy = timed_alone(lambda: R.check(R.rowsm_stream_copy(
            x.data_ptr(), y.data_ptr(), rows * 64, R.BF16, R.BF16, sh)), reps, flush, stream)
        out.append({"rows": rows, "cols": 64, "bytes": rows * 64 * 4,
                    "launch": R.rowsm_describe(rows, 64, R.BF16, R.BF16)[1],
                    "avg_us": kern, "copy_us": copy})
        del x, y
    return {"size_sweep": out, "launches_per_size": reps + 2}


def stream_overlap(pairs: int = 4):
    """Two exchanging launches of long rows on two streams that are never
    ordered against each other, issued in pairs (A on one stream, B on the
    other).  Each launch is capped at one block per compute unit (its groups
    loop over the rows), so it occupies part of every compute unit for a
    millisecond or more and the two streams' launches can run at the same
    time.  Every output is compared with the same launch made alone
    beforehand (bitwise).  A kernel trace of this run shows how much the two
    streams' dispatches overlap in time."""
    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    dev = torch.device("cuda:0")
    cfg = R.RowsmConfig(blocks_per_cu=1)
    xa = W.random_matrix(256, 262144, "f32", sigma=2.0, seed=1, device=dev)
    xb = W.random_matrix(512, 151936, "bf16", sigma=3.0, seed=2, device=dev)
    ya_ref = R.softmax(xa, config=cfg)
    yb_ref = R.softmax(xb, out_dtype=torch.float32, config=cfg)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    ya = [torch.empty_like(ya_ref) for _ in range(pairs)]
    yb = [torch.empty_like(yb_ref) for _ in range(pairs)]
    # one launch on each stream first, so that neither stream's first use
    # falls inside the pairs
    R.softmax(xa, out=ya[0], config=cfg, stream=s1)
    R.softmax(xb, out=yb[0], config=cfg, stream=s2)
    torch.cuda.synchronize()
    for i in range(pairs):
        R.softmax(xa, out=ya[i], config=cfg, stream=s1)
        R.softmax(xb, out=yb[i], config=cfg, stream=s2)
    torch.cuda.synchronize()
    same = all(torch.equal(a, ya_ref) for a in ya) and all(torch.equal(b, yb_ref) for b in yb)
    if not same or R.rowsm_split_wait_failures() != 0:
        raise R.RowsmError("two-stream launches differ from the same launches made alone")
    return {"stream_overlap": {
        "launch_a": R.rowsm_describe_op(R.OP_SOFTMAX, 256, 262144, R.F32, R.F32, cfg)[1],
        "launch_b": R.rowsm_describe_op(R.OP_SOFTMAX, 512, 151936, R.BF16, R.F32, cfg)[1],
        "rows_a": 256, "rows_b": 512, "pairs": pairs, "warm_up_launches": 2,
        "outputs_equal_to_launches_alone": same}}


def launcher_check(reps: int = 8):
    """The launcher's choice for launches of the shapes above against the
    other launch shapes of the library (medium wave groups with the default
    or one row per block, the single-read form with 1-4 blocks of 256 or 512
    threads; for rows of at most 256 columns the grid capped at 4-128 blocks
    per compute unit, blocks of 64 or 256 threads with 1 or 4 row groups per
    lane, and one-wave medium groups with the default or one row per block),
    each launch timed alone after a cache-evicting write.
    Every timed shape makes reps + 2 launches, in the order listed."""
    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    out = []
    for op, rows, cols, din, dout in LAUNCHER_SHAPES:
        print(f"launcher check: {op} {rows}x{cols} {din}->{dout}", file=sys.stderr, flush=True)
        if op == "backward":  # x holds probability rows, dy the upstream gradient
            x = W.random_probabilities(rows, cols, din, 0.3, seed=cols, device=dev)
            dy = W.random_matrix(rows, cols, din, sigma=1.0, seed=cols + 1, device=dev)
        else:
            x = W.random_matrix(rows, cols, din, sigma=3.0, seed=cols, device=dev)
        y = torch.empty(rows, cols, dtype=W.TORCH_DTYPES[dout], device=dev)
        if cols <= 256:
            alts = ([("auto", None)] +
                    [(f"bpc{b}", R.RowsmConfig(blocks_per_cu=b)) for b in (4, 8, 16, 64, 128)] +
                    [(f"b{b}r{r}", R.RowsmConfig(block=b, rows_per_lane=r))
                     for b, r in ((256, 4), (256, 1), (64, 1), (64, 4))] +
                    [("M1", R.RowsmConfig(variant=R.MEDIUM, waves_per_row=1)),
                     ("M1r1", R.RowsmConfig(variant=R.MEDIUM, waves_per_row=1,
                                            rows_per_block=1))])
        else:
            alts = ([("auto", None)] +
                    [(f"M{w}", R.RowsmConfig(variant=R.MEDIUM, waves_per_row=w))
                     for w in (1, 2, 4, 8, 16)] +
                    [(f"M{w}r1", R.RowsmConfig(variant=R.MEDIUM, waves_per_row=w,
                                               rows_per_block=1)) for w in (2, 4, 8)] +
                    [(f"S{S}T{T}", R.RowsmConfig(variant=R.LARGE, split_blocks=S, block=T))
                     for S in (1, 2, 4) for T in (256, 512)])
        code = {"scaled_causal": R.OP_SCALED_CAUSAL,
                "backward": R.OP_SOFTMAX_BACKWARD}.get(op, R.OP_SOFTMAX)
        rec = {"op": op, "rows": rows, "cols": cols, "in": din, "out": dout,
               "causal_period": cols if op == "scaled_causal" else 0,
               "launch": R.rowsm_describe_op(code, rows, cols, R.dtype_code(x.dtype),
                                             R.dtype_code(y.dtype))[1],
               "timed": [], "us": {}}
        for name, cfg in alts:
            def call(cfg=cfg):
                if op == "scaled_causal":
                    R.scaled_causal_softmax(x, 0.125, cols, 0, out=y, config=cfg)
                elif op == "backward":
                    R.softmax_backward(x, dy, out=y, config=cfg)
                else:
                    R.softmax(x, out=y, config=cfg)
            try:
                rec["us"][name] = timed_alone(call, reps, flush, stream)
            except R.RowsmError:
                continue  # a shape the family cannot take: refused, nothing launched
            rec["timed"].append(name)
        best = min(rec["us"], key=rec["us"].get)
        rec["best"] = best
        rec["auto_over_best"] = rec["us"]["auto"] / rec["us"][best]
        out.append(rec)
        del x, y
    if R.rowsm_split_wait_failures() != 0:
        raise R.RowsmError("split-row exchange waits gave up: results invalid")
    return {"launcher_check": out, "reps_per_shape": reps + 2}


# The calibration copy of the traffic counters: torch's device copy of 1 GiB
# (the runtime's copyBuffer kernel), run under rocprofv3 --pmc FETCH_SIZE and
# --pmc WRITE_SIZE.
CALIBRATION_BYTES = 1 << 30
CALIBRATION_COPY = ("import torch; a=torch.ones(1<<28, device='cuda'); b=torch.empty_like(a); "
                    "torch.cuda.synchronize(); [b.copy_(a) for _ in range(3)]; "
                    "torch.cuda.synchronize()")


def summarize(args) -> int:
    """Write profiles/ summaries from rocprofv3 CSV output (no GPU)."""
    import shlex

    import bench_profiles as P
    if not args.command.strip():
        print("a summary names the commands that made its rocprofv3 output: pass --command",
              file=sys.stderr)
        return 2
    # the header: the given commands, then this summariser's own invocation
    argv, skip = [], False
    for a in sys.argv[1:]:
        if skip:
            skip = False
        elif a == "--command":
            skip = True
        elif not a.startswith("--command="):
            argv.append(a)
    given = [ln for ln in args.command.strip().splitlines()
             if not ln.lstrip().startswith("python3 bench.py --summarize")]
    args.command = "\n".join(given + [
        "python3 bench.py " + " ".join(shlex.quote(a) for a in argv) +
        ' --command "<the lines above>"'])
    if args.summarize_trace:
        log, d, out = args.summarize_trace
        text = P.summarize_trace(log, d, args.command, PEAK_HBM_GBS)
    elif args.summarize_launcher:
        log, d, out = args.summarize_launcher
        text = P.summarize_launcher(log, d, args.command, PEAK_HBM_GBS)
    elif args.summarize_sweep:
        log, d, out = args.summarize_sweep
        text = P.summarize_sweep(log, d, args.command, PEAK_HBM_GBS)
    elif args.summarize_overlap:
        log, d, out = args.summarize_overlap
        text = P.summarize_overlap(log, d, args.command)
    elif args.summarize_pmc:
        log, d, out = args.summarize_pmc
        text = P.summarize_pmc(log, d, args.command)
    else:
        log, fd, wd, cfd, cwd, out, out_json = args.summarize_counters
        text, table = P.summarize_counters(log, fd, wd, cfd, cwd, CALIBRATION_BYTES,
                                           args.command, kernel_source_hash, kernel_family)
        with open(out_json, "w") as f:
            json.dump(table, f, indent=1)
            f.write("\n")
    with open(out, "w") as f:
        f.write(text)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--regimes", default=None,
                    help="comma-separated subset of the regimes (default: all four)")
    ap.add_argument("--no-next", action="store_true",
                    help="skip the measurements of the fused scale+causal form, "
                         "log-softmax, the softmax backward and the MoE group score")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="host threads of the CPU baseline (0 = every core this process may use)")
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="minimum seconds of oracle time for the CPU baseline (0 = skip)")
    ap.add_argument("--launcher-check", action="store_true",
                    help="instead of the step: time the launcher's choice for launches "
                         "of representative row lengths against the library's other launch "
                         "shapes, and print that as the JSON line")
    ap.add_argument("--size-sweep", action="store_true",
                    help="instead of the step: the small-row kernel and the plain copy at "
                         "4 MiB to 1 GiB, each launch alone (for a kernel trace)")
    ap.add_argument("--stream-overlap", action="store_true",
                    help="instead of the step: exchanging launches of few long rows on two "
                         "unordered streams, in pairs (for a kernel trace)")
    ap.add_argument("--summarize-overlap", nargs=3, metavar=("BENCH_LOG", "TRACE_DIR", "OUT_MD"),
                    help="no GPU: the overlap in time of the two streams' dispatches, from a "
                         "rocprofv3 --kernel-trace run of bench.py --stream-overlap")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="only run the calibration copy of the traffic counters "
                         "(CALIBRATION_COPY) and exit")
    ap.add_argument("--summarize-sweep", nargs=3, metavar=("BENCH_LOG", "TRACE_DIR", "OUT_MD"),
                    help="no GPU: the size-sweep summary from a rocprofv3 --kernel-trace run "
                         "of bench.py --size-sweep")
    ap.add_argument("--summarize-pmc", nargs=3, metavar=("BENCH_LOG", "PMC_DIR", "OUT_MD"),
                    help="no GPU: per-launch averages of every counter of a rocprofv3 --pmc "
                         "run of bench.py")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("BENCH_LOG", "TRACE_DIR", "OUT_MD"),
                    help="no GPU: write the kernel-trace summary of a rocprofv3 --kernel-trace "
                         "run of bench.py (its printed JSON line in BENCH_LOG)")
    ap.add_argument("--summarize-launcher", nargs=3,
                    metavar=("BENCH_LOG", "TRACE_DIR", "OUT_MD"),
                    help="no GPU: the same for a rocprofv3 run of bench.py --launcher-check")
    ap.add_argument("--summarize-counters", nargs=7,
                    metavar=("BENCH_LOG", "FETCH_DIR", "WRITE_DIR", "CAL_FETCH_DIR",
                             "CAL_WRITE_DIR", "OUT_MD", "OUT_JSON"),
                    help="no GPU: the HBM traffic summary and table from rocprofv3 --pmc "
                         "FETCH_SIZE and WRITE_SIZE runs of bench.py and of the calibration "
                         "copy (CALIBRATION_COPY)")
    ap.add_argument("--command", default="",
                    help="with --summarize-*: the command(s) that produced the rocprofv3 "
                         "output, written into the summary")
    args = ap.parse_args()

    if (args.summarize_trace or args.summarize_launcher or args.summarize_counters
            or args.summarize_sweep or args.summarize_pmc or args.summarize_overlap):
        return summarize(args)
    if args.calibration_copy:
        exec(CALIBRATION_COPY, {})
        return 0

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this row-softmax path runs on one GPU; rows shard across "
              "GPUs with no communication, so no multi-GPU run is made (use --gpus 1).",
              file=sys.stderr)
        return 2

    import torch

    import paper_2607_23089_amd as R
    from paper_2607_23089_amd import workloads as W

    R.lib()  # fails loudly when the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.launcher_check:
        print(json.dumps(launcher_check()), flush=True)
        return 0
    if args.size_sweep:
        print(json.dumps(size_sweep()), flush=True)
        return 0
    if args.stream_overlap:
        print(json.dumps(stream_overlap()), flush=True)
        return 0
    regimes = list(W.REGIMES if not args.regimes else args.regimes.split(","))

    inputs, outputs, calls = {}, {}, []
    stream = torch.cuda.current_stream(dev)
    for name in regimes:
        w = W.WORKLOADS[name]
        x = W.make_input(w, device=dev)
        y = torch.empty(w.rows, w.cols, dtype=W.TORCH_DTYPES[w.out_dtype], device=dev)
        inputs[name], outputs[name] = x, y
        calls.append((name, w, x.data_ptr(), y.data_ptr(), R.dtype_code(x.dtype),
                      R.dtype_code(y.dtype)))
    torch.cuda.synchronize()
    sh = stream.cuda_stream

    def step(events=None):
        for i, (name, w, xp, yp, di, do) in enumerate(calls):
            if events is not None:
                events[i][0].record(stream)
            st = R.rowsm_forward(xp, yp, w.rows, w.cols, di, do, sh)
            if st != R.OK:
                raise R.RowsmError(f"{name}: status {st} {R.rowsm_status_string(st)}")
            if events is not None:
                events[i][1].record(stream)

    def copy_step(events=None):
        # The library's streaming copy of each regime's bytes (same dtype
        # pair, same buffers): what a plain copy of the same bytes takes.
        for i, (name, w, xp, yp, di, do) in enumerate(calls):
            if events is not None:
                events[i][0].record(stream)
            st = R.rowsm_stream_copy(xp, yp, w.rows * w.cols, di, do, sh)
            if st != R.OK:
                raise R.RowsmError(f"copy {name}: status {st} {R.rowsm_status_string(st)}")
            if events is not None:
                events[i][1].record(stream)

    # Parity gate: one untimed step, its outputs checked against the oracle on
    # sampled rows of every regime before anything is timed.  A failure ends
    # the run with no value.
    step()
    torch.cuda.synchronize()
    gate = parity_gate(inputs, outputs, regimes, args.cpu_threads)
    gate_ok = all(g["parity_ok"] for g in gate.values())
    if R.rowsm_split_wait_failures() != 0:
        gate_ok = False
    if not gate_ok:
        print("bench.py: parity gate failed, nothing timed: " + json.dumps(gate),
              file=sys.stderr)
        print(json.dumps({"metric": METRIC, "value": None, "unit": "GB/s", "n_gpus": 1,
                          "parity_gate": gate}), flush=True)
        return 1

    for _ in range(args.warmup):
        step()
        copy_step()
    torch.cuda.synchronize()

    # Copies first, so that the timed softmax steps leave their
    # outputs in y for the CPU baseline's parity check.
    cevs = [[[HipEvent() for _ in range(2)] for _ in calls] for _ in range(args.steps)]
    torch.cuda.synchronize()
    copy_step()  # untimed: the timed launches start on a busy device
    for k in range(args.steps):
        copy_step(cevs[k])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        copy_step()
    torch.cuda.synchronize()
    copy_wall = time.perf_counter() - t0

    # Per-launch times: the steps with a HIP event pair around each launch.
    evs = [[[HipEvent() for _ in range(2)] for _ in calls]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    step()  # untimed: the timed launches start on a busy device
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    # Whole-step throughput: the same steps again, without the per-launch
    # events (their markers sit between the kernels), timed by the host
    # clock between two device synchronisations.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    step_bytes = sum(W.WORKLOADS[n].algorithmic_bytes for n in regimes)
    ms_per_step = wall / args.steps * 1e3
    per = {}
    for i, (name, w, *_r) in enumerate(calls):
        ms = [evs[k][i][0].elapsed_time(evs[k][i][1]) for k in range(args.steps)]
        ms.sort()
        avg = sum(ms) / len(ms)
        gbs = w.algorithmic_bytes / (avg * 1e-3) / 1e9
        st, desc = R.rowsm_describe(w.rows, w.cols, R.dtype_code(W.TORCH_DTYPES[w.in_dtype]),
                                    R.dtype_code(W.TORCH_DTYPES[w.out_dtype]))
        cavg = sum(cevs[k][i][0].elapsed_time(cevs[k][i][1]) for k in range(args.steps)) \
            / args.steps
        cgbs = w.algorithmic_bytes / (cavg * 1e-3) / 1e9
        per[name] = {
            "kernel": desc.split(" ")[0], "launch": desc,
            "algorithmic_bytes": w.algorithmic_bytes,
            "avg_us": avg * 1e3, "median_us": ms[len(ms) // 2] * 1e3,
            "min_us": ms[0] * 1e3, "p10_us": ms[len(ms) // 10] * 1e3,
            "p90_us": ms[(9 * len(ms)) // 10] * 1e3,
            "GBps": gbs, "frac_of_peak": gbs / PEAK_HBM_GBS,
            "hbm_bytes_per_launch": measured_traffic(name, desc),
            "copy_us": cavg * 1e3, "copy_GBps": cgbs, "ratio_to_copy": gbs / cgbs,
            "target_frac_of_peak": TARGET_FRAC.get(name),
            "meets_target": (gbs / PEAK_HBM_GBS >= TARGET_FRAC[name]) if name in TARGET_FRAC
            else None,
        }
    failures = R.rowsm_split_wait_failures()
    if failures != 0:
        raise R.RowsmError(f"{failures} split-row exchange waits gave up: results invalid")
    mem = device_memory_info(torch.cuda.current_device())
    hbm_info = dict(mem, spec_peak_GBps=PEAK_HBM_GBS)
    if mem.get("memory_clock_khz") and mem.get("bus_width_bits"):
        # bytes per second the reported clock and width give at one transfer
        # per pin per clock; the per-pin data rate the spec peak implies
        one = mem["memory_clock_khz"] * 1e3 * mem["bus_width_bits"] / 8 / 1e9
        hbm_info["GBps_at_one_transfer_per_clock"] = one
        hbm_info["transfers_per_clock_at_spec_peak"] = PEAK_HBM_GBS / one
    dom = max(per, key=lambda n: per[n]["avg_us"])
    d = per[dom]
    value = step_bytes / (wall / args.steps) / 1e9

    result = {
        "metric": METRIC,
        "value": value,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded, generated on the GPU)",
        "config": {
            "workload": "row softmax over the row-length regimes, one launch each per step: "
                        + ", ".join(f"{n} {W.WORKLOADS[n].in_dtype}->{W.WORKLOADS[n].out_dtype}"
                                    for n in regimes),
            "algorithmic_bytes_per_step": step_bytes,
            "regimes": {n: {"GBps": round(v["GBps"], 1),
                            "frac_of_peak": round(v["frac_of_peak"], 4),
                            "avg_us": round(v["avg_us"], 2), "kernel": v["kernel"],
                            "ratio_to_copy": round(v["ratio_to_copy"], 4),
                            "target_frac_of_peak": v["target_frac_of_peak"],
                            "meets_target": v["meets_target"]}
                        for n, v in per.items()},
        },
        "roofline": {
            "bound": "hbm",
            "kernel": f"{d['kernel']} ({dom})",
            "achieved": d["GBps"],
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": d["GBps"] / PEAK_HBM_GBS,
            "traffic": d["hbm_bytes_per_launch"],
            "algorithmic_bytes_per_launch": d["algorithmic_bytes"],
            "avg_launch_us": d["avg_us"],
            "copy_GBps": d["copy_GBps"],
            "ratio_to_copy": d["ratio_to_copy"],
        },
        "copy_step": {
            "what": "the library's streaming copy (rowsm_stream_copy) of each regime's bytes, "
                    "same dtype pairs and buffers, back to back in the same protocol",
            "GBps": step_bytes / (copy_wall / args.steps) / 1e9,
            "ms_per_step": copy_wall / args.steps * 1e3,
        },
        "regimes_detail": per,
        "parity_gate": {"parity_ok": gate_ok,
                        "max_tol_ratio": max(g["max_tol_ratio"] for g in gate.values()),
                        "when": "before timing, on the outputs of one untimed step",
                        "regimes": gate},
        "device_hbm": hbm_info,
    }
    # The same step captured into a HIP graph and replayed (the single-read
    # form keeps its one-read plan under capture).
    graph_leg = None
    if not args.no_next:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            sh_cap = side.cuda_stream
            for name, w, xp, yp, di, do in calls:
                st = R.rowsm_forward(xp, yp, w.rows, w.cols, di, do, sh_cap)
                if st != R.OK:
                    raise R.RowsmError(f"capture {name}: status {st}")
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            g.replay()
        torch.cuda.synchronize()
        gwall = time.perf_counter() - t0
        graph_leg = {"what": "the step's four launches captured into one HIP graph, "
                             "replayed back to back",
                     "GBps": step_bytes / (gwall / args.steps) / 1e9,
                     "ms_per_step": gwall / args.steps * 1e3}
        del g
        if R.rowsm_split_wait_failures() != 0:
            raise R.RowsmError("split-row exchange waits gave up under graph replay")
    if graph_leg is not None:
        result["graph_step"] = graph_leg
    if not args.no_next:
        result["context"] = copy_ceiling()
        result["launch_bound"] = launch_bound_leg(reps=20)
        result["next_rows"] = {"fused_scale_causal": fused_causal_leg(reps=10),
                               "log_softmax": log_softmax_leg(reps=10),
                               "softmax_backward": backward_leg(reps=10),
                               "moe_group_top2": moe_leg(reps=10)}
    if args.cpu_budget > 0:
        cb = cpu_baseline(inputs, outputs, regimes, args.cpu_budget, args.cpu_threads)
        cb["parity_ok"] = all(p["parity_ok"] for p in cb["parity_on_sample"].values())
        cb["max_tol_ratio"] = max(p["max_tol_ratio"] for p in cb["parity_on_sample"].values())
        result["cpu_baseline"] = cb
        if not cb["parity_ok"]:
            print("bench.py: the timed steps' outputs fail parity on the CPU baseline's "
                  "rows: " + json.dumps(cb["parity_on_sample"]), file=sys.stderr)
            result["value"] = None
            print(json.dumps(result), flush=True)
            return 1
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
