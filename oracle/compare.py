"""Parity comparator: GPU row-softmax output vs the fp64 oracle.

TEST INFRASTRUCTURE ONLY (same rule as the rest of ``oracle/``).

Rules (the oracle value ``v`` is fp64 and is never rounded to the output
dtype first; ``y`` is the GPU output widened exactly to fp64):

  * NaN pattern: ``isnan(y) == isnan(v)`` at every position.
  * ``v == 0`` (masked -inf entries, fp64 underflow): ``y`` must be +-0.
  * fp32 output: ``|y - v| <= 2e-6``.
  * bf16 output: ``|y - v| <= ulp_bf16(v)`` with
    ``ulp_bf16(v) = 2**(max(floor(log2|v|), -126) - 7)``, the spacing of bf16
    numbers in v's binade; for ``|v| < 2**-126`` a difference up to ``2**-126``
    is also accepted (flush of a subnormal result to zero).

The maximum relative error over entries with ``|v| >= 1e-30`` is reported but
does not gate.
"""
from __future__ import annotations

import numpy as np

F32_ABS_TOL = 2e-6
BF16_SUBNORMAL_SLACK = 2.0 ** -126


def ulp_bf16(v: np.ndarray) -> np.ndarray:
    """Spacing of bf16 numbers in the binade of each |v| (v != 0)."""
    a = np.abs(np.asarray(v, dtype=np.float64))
    _, e = np.frexp(a)                      # a = f * 2**e, f in [0.5, 1)
    ex = np.maximum(e.astype(np.int64) - 1, -126)
    return np.ldexp(1.0, (ex - 7).astype(np.int32))


def widen_output(y: np.ndarray, out_dtype: str) -> np.ndarray:
    """GPU output -> fp64, exact.  ``y`` is fp32 values for 'f32', or bf16 bit
    patterns (uint16/int16) for 'bf16'."""
    if out_dtype == "f32":
        return np.asarray(y, dtype=np.float32).astype(np.float64)
    if out_dtype == "bf16":
        u = np.asarray(y).view(np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown out_dtype {out_dtype!r}")


def compare(y: np.ndarray, v: np.ndarray, out_dtype: str) -> dict:
    """Check GPU output ``y`` (already widened to fp64) against oracle ``v``.

    Returns a dict with ``ok`` and the statistics; ``worst`` is the flat index
    of the largest tolerance ratio (None when everything is exact)."""
    y = np.asarray(y, dtype=np.float64).ravel()
    v = np.asarray(v, dtype=np.float64).ravel()
    if y.shape != v.shape:
        raise ValueError(f"shape mismatch {y.shape} vs {v.shape}")
    ny, nv = np.isnan(y), np.isnan(v)
    nan_mismatch = int(np.count_nonzero(ny != nv))
    fin = ~(ny | nv)
    zero = fin & (v == 0.0)
    zero_mismatch = int(np.count_nonzero(zero & (y != 0.0)))
    diff = np.where(fin, np.abs(y - v), 0.0)
    if out_dtype == "f32":
        tol = np.full_like(v, F32_ABS_TOL)
    elif out_dtype == "bf16":
        tol = np.where(v != 0.0, ulp_bf16(np.where(v != 0.0, v, 1.0)), 0.0)
        tol = np.where(np.abs(v) < 2.0 ** -126,
                       np.maximum(tol, BF16_SUBNORMAL_SLACK), tol)
        tol = np.where(zero, 0.0, tol)
    else:
        raise ValueError(f"unknown out_dtype {out_dtype!r}")
    over = fin & (diff > tol)
    n_over = int(np.count_nonzero(over))
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(fin & (tol > 0), diff / np.where(tol > 0, tol, 1.0), 0.0)
        big = fin & (np.abs(v) >= 1e-30)
        rel = np.where(big, diff / np.where(big, np.abs(v), 1.0), 0.0)
    worst = int(np.argmax(ratio)) if ratio.size and ratio.max() > 0 else None
    return {
        "ok": nan_mismatch == 0 and zero_mismatch == 0 and n_over == 0,
        "n": int(v.size),
        "max_abs": float(diff.max()) if diff.size else 0.0,
        "max_tol_ratio": float(ratio.max()) if ratio.size else 0.0,
        "max_rel": float(rel.max()) if rel.size else 0.0,
        "n_over_tol": n_over,
        "nan_mismatch": nan_mismatch,
        "zero_mismatch": zero_mismatch,
        "worst": worst,
    }


# ---------------------------------------------------------------------------
# Log-softmax outputs.
#
# The GPU computes y = (x - m) - ln(s) in fp32, m the row maximum and
# s = sum 2^((x - m') log2e) taken relative to m (or, in the two-pass form,
# to a reference m' <= m that trails the running maximum by at most 8, and
# rescaled to m at the end of each thread's pass).  Error sources, u = 2^-24,
# for every row length the library accepts (n < 2^30):
#   * the roundings of x - m and of the final difference: <= 2u |v| in all
#     (|x - m| <= |v| because ln(s) >= 0);
#   * the relative error of s:
#       exponentials: v_exp_f32 (1 ulp, <= 2u) and the two roundings of its
#       argument a, which a term carries as <= 1.4u |a|; weighted by the
#       terms, |a| averages at most log2(n) + 1.5 (+ 11.5 for the trailing
#       reference), so <= 2u + 1.4u * 43 ~= 62u;
#       additions: a lane's serial chain of at most 64 terms (register-
#       resident forms) or one tile of <= 32 terms plus a Kahan-compensated
#       sum over tiles (2u + t u^2 <= 2.5u for t <= 2^23 tiles: independent
#       of the row length), then 6 lane levels, <= 15 waves in order and, for
#       several blocks per row, <= 3 + 6 levels: <= 94u;
#       rescales (<= 4u each): the two-pass form's reference moves (their
#       errors are damped by e^-8 per later move, <= 13u in all), the
#       rescale to m (4u), and one per merge level (lane, wave, block: <= 16u):
#       <= 33u;
#     in all <= 189u ~= 1.13e-5;
#   * v_log_f32 (1 ulp of log2 s) and the multiplication by ln 2:
#     <= 2^-23 ln(s) + u ln(s) <= 3.7e-6 for s <= 2^30.
# These first-order worst cases add up to 1.5e-5 + 2u |v|; the fp32 bound is
# 2e-5 + 2^-22 |v|.  A bf16 output adds one bf16 ulp of v (round to nearest
# of a value already within the fp32 bound).

LOG_ABS_TOL = 2e-5
LOG_REL_TOL = 2.0 ** -22
_OVERFLOW = {"f32": 2.0 ** 128 * (1 - 2.0 ** -25), "bf16": 2.0 ** 128 * (1 - 2.0 ** -9)}


def compare_log(y: np.ndarray, v: np.ndarray, out_dtype: str) -> dict:
    """Check a GPU log-softmax output ``y`` (widened to fp64) against the
    oracle ``v``: NaN positions equal; -inf exactly where ``v`` rounds to -inf
    in the output dtype; elsewhere ``|y - v| <= 2e-5 + 2^-22 |v|`` (fp32)
    plus one bf16 ulp of v (bf16)."""
    y = np.asarray(y, dtype=np.float64).ravel()
    v = np.asarray(v, dtype=np.float64).ravel()
    if y.shape != v.shape:
        raise ValueError(f"shape mismatch {y.shape} vs {v.shape}")
    if out_dtype not in _OVERFLOW:
        raise ValueError(f"unknown out_dtype {out_dtype!r}")
    ny, nv = np.isnan(y), np.isnan(v)
    nan_mismatch = int(np.count_nonzero(ny != nv))
    v_inf = np.isinf(v) | (np.abs(np.where(nv, 0.0, v)) >= _OVERFLOW[out_dtype])
    v_out = np.where(v_inf & ~nv, np.copysign(np.inf, v), v)
    inf_mismatch = int(np.count_nonzero((np.isinf(y) | np.isinf(v_out)) & ~(ny | nv)
                                        & (y != v_out)))
    fin = ~(ny | nv | np.isinf(y) | np.isinf(v_out))
    with np.errstate(invalid="ignore"):
        diff = np.where(fin, np.abs(y - v), 0.0)
    tol = LOG_ABS_TOL + LOG_REL_TOL * np.abs(np.where(fin, v, 0.0))
    if out_dtype == "bf16":
        tol = tol + np.where(fin & (v != 0.0), ulp_bf16(np.where(fin & (v != 0.0), v, 1.0)), 0.0)
    over = fin & (diff > tol)
    ratio = np.where(fin, diff / tol, 0.0)
    worst = int(np.argmax(ratio)) if ratio.size and ratio.max() > 0 else None
    return {
        "ok": nan_mismatch == 0 and inf_mismatch == 0 and not over.any(),
        "n": int(v.size),
        "max_abs": float(diff.max()) if diff.size else 0.0,
        "max_tol_ratio": float(ratio.max()) if ratio.size else 0.0,
        "n_over_tol": int(np.count_nonzero(over)),
        "nan_mismatch": nan_mismatch,
        "inf_mismatch": inf_mismatch,
        "worst": worst,
    }


# ---------------------------------------------------------------------------
# Softmax-backward outputs.
#
# The GPU computes d = sum_k y_k dy_k with fma in fp32: a lane's chain of at
# most 64 products in the register-resident forms, or, in the two-pass form,
# one tile of <= 32 products plus a Kahan-compensated sum over the tiles
# (2u + t u^2 <= 2.5u for t <= 2^23 tiles, so the row length does not enter);
# then a lane tree of depth 6, at most 16 waves in order and, for several
# blocks per row, <= 3 + 6 levels.  So |d_gpu - d| <= 94u S <= 128u S with
# S = sum_k |y_k dy_k| and u = 2^-24 (first order), for every row length the
# library accepts.  Then dx_j = y_j * (dy_j - d_gpu) adds two roundings.
# Hence, per element,
#     |dx_gpu - dx| <= |y_j| (2^-17 S + 2^-23 |dy_j - d|) + 2^-23 |dx_j|
# (the single roundings doubled for margin), plus 2^-126 where the result is
# below the normal range (a flushed subnormal), plus one bf16 ulp of dx_j for
# bf16 output.  y_j == 0 must give an exact zero.

BWD_DOT_REL = 2.0 ** -17
BWD_ROUND = 2.0 ** -23


def compare_backward(dx: np.ndarray, v: np.ndarray, y: np.ndarray, dy: np.ndarray,
                     out_dtype: str) -> dict:
    """Check a GPU softmax-backward output ``dx`` (widened to fp64) against the
    oracle ``v``, given the fp64-widened inputs ``y`` and ``dy`` (rows x cols)."""
    y = np.asarray(y, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    rows, cols = y.shape
    dx = np.asarray(dx, dtype=np.float64).reshape(rows, cols)
    v = np.asarray(v, dtype=np.float64).reshape(rows, cols)
    if out_dtype not in ("f32", "bf16"):
        raise ValueError(f"unknown out_dtype {out_dtype!r}")
    ny, nv = np.isnan(dx), np.isnan(v)
    nan_mismatch = int(np.count_nonzero(ny != nv))
    inf_mismatch = int(np.count_nonzero((np.isinf(dx) | np.isinf(v)) & ~(ny | nv) & (dx != v)))
    fin = np.isfinite(dx) & np.isfinite(v)
    with np.errstate(invalid="ignore", over="ignore"):
        S = np.sum(np.abs(y * dy), axis=1, keepdims=True)
        d = np.sum(y * dy, axis=1, keepdims=True)
        tol = np.abs(y) * (BWD_DOT_REL * S + BWD_ROUND * np.abs(dy - d)) + BWD_ROUND * np.abs(v)
    tol = np.where(np.isfinite(tol), tol, np.inf)
    tol = np.where(np.abs(v) < 2.0 ** -126, np.maximum(tol, 2.0 ** -126), tol)
    if out_dtype == "bf16":
        nz = fin & (v != 0.0)
        tol = tol + np.where(nz, ulp_bf16(np.where(nz, v, 1.0)), 0.0)
    zero = fin & (y == 0.0)
    zero_mismatch = int(np.count_nonzero(zero & (dx != 0.0)))
    with np.errstate(invalid="ignore"):
        diff = np.where(fin, np.abs(dx - v), 0.0)
    over = fin & (diff > tol)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(fin & (tol > 0), diff / np.where(tol > 0, tol, 1.0), 0.0)
    worst = int(np.argmax(ratio)) if ratio.size and ratio.max() > 0 else None
    return {
        "ok": nan_mismatch == 0 and inf_mismatch == 0 and zero_mismatch == 0 and not over.any(),
        "n": int(v.size),
        "max_abs": float(diff.max()) if diff.size else 0.0,
        "max_tol_ratio": float(ratio.max()) if ratio.size else 0.0,
        "n_over_tol": int(np.count_nonzero(over)),
        "nan_mismatch": nan_mismatch,
        "inf_mismatch": inf_mismatch,
        "zero_mismatch": zero_mismatch,
        "worst": worst,
    }
