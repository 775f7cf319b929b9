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
