"""fp64 CPU oracle for row softmax -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library never imports, links or
calls it, and it never imports the HIP library: the two share no code.

Contents
  * ``softmax_f64``   -- the oracle proper, a plain C loop (``softmax_f64.c``)
                         over fp64 rows: max, exp(x - max), sequential sum,
                         divide.  That is the textbook stable softmax over the
                         last dimension, which is what PyTorch's reference
                         computes (the paper judges every operator against a
                         PyTorch reference: Evaluation, Experimental Setup).
  * ``softmax_scaled_causal_f64`` -- the same definition applied to
                         scale * x with a causal mask from the indices
                         (scaled attention scores).
  * ``log_softmax_f64``  -- x - max - log(sum exp(x - max)) per row.
  * ``softmax_backward_f64`` -- dx = y * (dy - sum(y * dy)) per row, the
                         softmax Jacobian applied to dy.
  * ``moe_group_top2_f64`` -- the paper's running example (``moe_group_f64.c``):
                         per group of G consecutive expert scores, the sum of
                         its two largest values (a tied maximum counts twice),
                         an fp32 sum rounded to the output dtype.
  * ``widen_f32`` / ``widen_bf16_bits`` -- exact widening of the stored input
                         bit patterns to fp64 (bf16 -> bits << 16 -> fp32 ->
                         fp64), so the oracle sees exactly the values the GPU
                         reads.
  * ``build``         -- compiles ``softmax_f64.c`` with gcc (``build_moe``:
                         ``moe_group_f64.c``).

The oracle is pinned by tests/test_oracle.py (high-precision brute force with a
different formula, closed forms, invariants, library routines) and
tests/test_oracle_mutants.py (planted mistakes must fail those pins).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "softmax_f64.c")
_LIB = os.path.join(_HERE, "liboracle_softmax.so")

_MOE_SRC = os.path.join(_HERE, "moe_group_f64.c")
_MOE_LIB = os.path.join(_HERE, "liboracle_moe.so")

_lib = None
_moe_lib = None


def gcc_command(src: str, out: str) -> list:
    """The gcc line that builds the oracle (IEEE semantics: no fast-math, no
    contraction of a*b+c into fma)."""
    return ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math",
            "-fPIC", "-shared", "-Wall", "-Wextra", "-Werror", "-o", out, src,
            "-lm", "-lpthread"]


def build(src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle's C source into a shared library; returns its path."""
    tmp = out + ".tmp"
    subprocess.run(gcc_command(src, tmp), check=True)
    os.replace(tmp, out)
    return out


def load(path: str | None = None):
    """Load (building first if absent) the oracle library; returns the
    ctypes handle with ``oracle_softmax_f64`` typed."""
    global _lib
    if path is None:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB):
            build()
        path = _LIB
    lib = ctypes.CDLL(path)
    fn = lib.oracle_softmax_f64
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.c_int64, ctypes.c_int]
    fn = lib.oracle_log_softmax_f64
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.c_int64, ctypes.c_int]
    fn = lib.oracle_softmax_backward_f64
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.c_int64, ctypes.c_int]
    fn = lib.oracle_softmax_scaled_causal_f64
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.c_int64, ctypes.c_double, ctypes.c_int64,
                   ctypes.c_int64, ctypes.c_int]
    if path == _LIB:
        _lib = lib
    return lib


def build_moe(src: str = _MOE_SRC, out: str = _MOE_LIB) -> str:
    """Compile the MoE group-score oracle; returns the library path."""
    return build(src, out)


def load_moe(path: str | None = None):
    """Load (building first if absent) the MoE group-score oracle library."""
    global _moe_lib
    if path is None:
        if _moe_lib is not None:
            return _moe_lib
        if not os.path.exists(_MOE_LIB):
            build_moe()
        path = _MOE_LIB
    lib = ctypes.CDLL(path)
    fn = lib.oracle_moe_group_top2_f64
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                   ctypes.c_int64, ctypes.c_int]
    if path == _MOE_LIB:
        _moe_lib = lib
    return lib


def moe_group_top2_f64(scores: np.ndarray, group: int, out_dtype: str = "f32",
                       lib=None) -> np.ndarray:
    """tokens x experts scores (fp64 values of the stored scores) ->
    tokens x (experts / group) group scores, each the fp32 sum of the group's
    two largest values rounded to ``out_dtype`` ('f32' or 'bf16'), as fp64."""
    s = np.ascontiguousarray(np.asarray(scores, dtype=np.float64))
    if s.ndim == 1:
        s = s[None, :]
    tokens, experts = s.shape
    if group < 2 or experts % group:
        raise ValueError("group must be >= 2 and divide the expert count")
    out = np.full((tokens, experts // group), np.nan)
    lib = lib if lib is not None else load_moe()
    rc = lib.oracle_moe_group_top2_f64(s.ctypes.data, out.ctypes.data, tokens, experts,
                                       int(group), 1 if out_dtype == "bf16" else 0)
    if rc != 0:
        raise RuntimeError(f"oracle_moe_group_top2_f64 failed with status {rc}")
    return out


def softmax_f64(x: np.ndarray, threads: int = 1, lib=None) -> np.ndarray:
    """y = softmax(x, axis=-1) in fp64 for a 2-D array (any leading shape is
    flattened to rows).  ``threads`` splits rows across host threads; the
    result does not depend on it."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if x.ndim == 1:
        x = x[None, :]
    shape = x.shape
    x2 = x.reshape(int(np.prod(shape[:-1])), shape[-1])
    y = np.full_like(x2, np.nan)  # rows the C code never writes stay NaN
    lib = lib if lib is not None else load()
    rc = lib.oracle_softmax_f64(x2.ctypes.data, y.ctypes.data, x2.shape[0],
                                x2.shape[1], int(threads))
    if rc != 0:
        raise RuntimeError(f"oracle_softmax_f64 failed with status {rc}")
    return y.reshape(shape)


def log_softmax_f64(x: np.ndarray, threads: int = 1, lib=None) -> np.ndarray:
    """y = log_softmax(x, axis=-1) in fp64 (2-D, rows x cols)."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if x.ndim == 1:
        x = x[None, :]
    y = np.full_like(x, np.nan)
    lib = lib if lib is not None else load()
    rc = lib.oracle_log_softmax_f64(x.ctypes.data, y.ctypes.data, x.shape[0], x.shape[1],
                                    int(threads))
    if rc != 0:
        raise RuntimeError(f"oracle_log_softmax_f64 failed with status {rc}")
    return y


def softmax_backward_f64(y: np.ndarray, dy: np.ndarray, threads: int = 1,
                         lib=None) -> np.ndarray:
    """dx = y * (dy - rowsum(y * dy)) in fp64 (2-D, rows x cols)."""
    y = np.ascontiguousarray(np.asarray(y, dtype=np.float64))
    dy = np.ascontiguousarray(np.asarray(dy, dtype=np.float64))
    if y.ndim == 1:
        y, dy = y[None, :], dy[None, :]
    if y.shape != dy.shape:
        raise ValueError("y and dy must have the same shape")
    dx = np.full_like(y, np.nan)
    lib = lib if lib is not None else load()
    rc = lib.oracle_softmax_backward_f64(y.ctypes.data, dy.ctypes.data, dx.ctypes.data,
                                         y.shape[0], y.shape[1], int(threads))
    if rc != 0:
        raise RuntimeError(f"oracle_softmax_backward_f64 failed with status {rc}")
    return dx


def softmax_scaled_causal_f64(x: np.ndarray, scale: float, period: int, offset: int,
                              threads: int = 1, lib=None, row0: int = 0) -> np.ndarray:
    """y = softmax(scale * x + mask) per row, mask(r, c) = -inf where
    period > 0 and c > ((row0 + r) mod period) + offset (row0: index of the
    first given row in the full matrix, so that samples keep their mask)."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if x.ndim == 1:
        x = x[None, :]
    rows, cols = x.shape
    y = np.full_like(x, np.nan)
    lib = lib if lib is not None else load()
    if row0 == 0:
        rc = lib.oracle_softmax_scaled_causal_f64(x.ctypes.data, y.ctypes.data, rows, cols,
                                                  float(scale), int(period), int(offset),
                                                  int(threads))
    else:  # shift the offset so row r sees its row0 + r query
        rc = 0
        for r in range(rows):
            q = (row0 + r) % period if period > 0 else 0
            rc |= lib.oracle_softmax_scaled_causal_f64(
                x[r].ctypes.data, y[r].ctypes.data, 1, cols, float(scale), 1 if period > 0 else 0,
                q + int(offset) if period > 0 else 0, 1)
    if rc != 0:
        raise RuntimeError(f"oracle_softmax_scaled_causal_f64 failed with status {rc}")
    return y


def widen_f32(x: np.ndarray) -> np.ndarray:
    """fp32 values -> fp64, exact."""
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def widen_bf16_bits(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16/int16) -> fp64, exact: the 16 bits are the
    high half of an fp32 word."""
    u = np.asarray(bits).view(np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)
