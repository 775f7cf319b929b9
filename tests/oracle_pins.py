"""Pins for the fp64 softmax oracle: facts fixed by mathematics, not by the
oracle's own code.

``run_pins(sm)`` applies every pin to a candidate implementation
``sm(x, threads=1) -> y`` (fp64 2-D arrays, softmax over the last axis) and
returns the list of failures.  The real oracle must return none
(tests/test_oracle.py); every planted mistake must trip at least one
(tests/test_oracle_mutants.py).

Pins
  brute_force   y_i = 1 / sum_j exp(x_j - x_i) in 50-digit mpmath: a different
                formula (no max subtraction, no division of a sum) evaluated
                far above fp64 precision, on tiny seeded inputs including ties,
                bf16-representable values, large spreads and -inf entries.
  closed_forms  hand-derived values (tests/golden/closed_forms.json).
  invariants    rows sum to 1; exact shift invariance on a coarse grid; a
                constant row gives exactly 1/C; a dominant entry gives exactly
                one-hot; -inf gives exactly 0; 0 <= y <= 1; order preserved;
                permutation equivariance; C == 1 gives 1; independence of
                the thread count; special rows (NaN, +inf, all -inf) are NaN.
  libraries     scipy.special.softmax and torch.softmax in fp64, both
                independent implementations of the same definition.
  orientation   a non-square matrix is normalised along rows, not columns.
"""
from __future__ import annotations

import json
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                      "closed_forms.json")


def _num(v):
    return float(v) if not isinstance(v, str) else float(v)


def brute_force_rows(x: np.ndarray) -> np.ndarray:
    """softmax by y_i = 1 / sum_j exp(x_j - x_i) at 50 decimal digits."""
    import mpmath
    mpmath.mp.dps = 50
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    for r in range(x.shape[0]):
        row = [mpmath.mpf(float(v)) for v in x[r]]
        for i, xi in enumerate(row):
            if mpmath.isinf(xi) and xi < 0:
                out[r, i] = 0.0
                continue
            tot = mpmath.mpf(0)
            for xj in row:
                if mpmath.isinf(xj) and xj < 0:
                    continue
                tot += mpmath.exp(xj - xi)
            out[r, i] = float(1 / tot)
    return out


def brute_force_inputs() -> list:
    """Tiny seeded inputs: several widths and spreads, ties, values on the
    bf16 grid, and -inf entries in rows that keep a finite maximum."""
    rng = np.random.default_rng(20260726)
    cases = []
    for cols in (1, 2, 3, 7, 8, 16, 33):
        for sigma in (1.0, 8.0, 100.0):
            x = rng.normal(0.0, sigma, size=(4, cols))
            if cols >= 3:
                x[1, cols // 2] = x[1, 0]                   # tie at an interior value
                x[2, :] = np.round(x[2, :], 0)              # many ties
                x[3, -1] = -np.inf                          # masked entry
            cases.append(x)
    # values representable in bf16 (8 significant bits)
    b = rng.normal(0.0, 4.0, size=(6, 16))
    m, e = np.frexp(b)
    cases.append(np.ldexp(np.round(m * 256.0) / 256.0, e))
    return cases


def _close(a, b, rel, abs_=0.0):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if a.shape != b.shape:
        return False
    na, nb = np.isnan(a), np.isnan(b)
    if not np.array_equal(na, nb):
        return False
    f = ~na
    return bool(np.all(np.abs(a[f] - b[f]) <= rel * np.abs(b[f]) + abs_))


def run_pins(sm) -> list:
    fails = []

    def fail(name, msg):
        fails.append(f"{name}: {msg}")

    # --- brute force -----------------------------------------------------
    for x in brute_force_inputs():
        try:
            y = sm(x)
        except Exception as e:  # a crashing candidate fails the pin
            fail("brute_force", f"raised {e!r}")
            break
        v = brute_force_rows(x)
        # fp64 error bound of exp(x - m) / s: the exponent's rounding is
        # amplified by |x - m| (conditioning of exp), each of the C terms of
        # the sum adds at most one rounding, and exp, the subtraction and the
        # division add a few more.
        with np.errstate(invalid="ignore"):
            gap = np.abs(x - np.max(np.where(np.isneginf(x), np.nan, x), axis=1,
                                    keepdims=True, initial=-np.inf, where=~np.isneginf(x)))
        gap = np.where(np.isfinite(gap), gap, 0.0)
        rel = (8.0 + 2.0 * gap + x.shape[1]) * 2.0 ** -53
        y = np.asarray(y, dtype=np.float64)
        ok = y.shape == v.shape and np.array_equal(np.isnan(y), np.isnan(v))
        if ok:
            ok = bool(np.all(np.abs(y - v) <= rel * np.abs(v) + 2.0 ** -1070))
        if not ok:
            d = np.abs(y - v) if y.shape == v.shape else np.array([np.nan])
            err = float(np.max(d[np.isfinite(d)])) if np.isfinite(d).any() else float("nan")
            fail("brute_force", f"shape {x.shape}: max abs diff {err:.3e}")

    # --- closed forms ----------------------------------------------------
    with open(GOLDEN) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        x = np.array([[_num(v) for v in case["x"]]])
        want = np.array([[_num(v) for v in case["y"]]])
        y = sm(x)
        tol = float(case["rel_tol"])
        ok = _close(y, want, tol) if tol > 0 else (
            np.array_equal(np.isnan(y), np.isnan(want))
            and np.array_equal(y[~np.isnan(y)], want[~np.isnan(want)]))
        if not ok:
            fail("closed_forms", f"{case['name']}: got {y.ravel().tolist()}")

    rng = np.random.default_rng(7)
    # --- invariants ------------------------------------------------------
    x = rng.normal(0.0, 3.0, size=(16, 129))
    y = sm(x)
    if not np.all(np.abs(y.sum(axis=1) - 1.0) <= x.shape[1] * 2.0 ** -52):
        fail("sum_to_one", f"max |sum-1| {np.max(np.abs(y.sum(axis=1) - 1.0)):.3e}")
    if not (np.all(y >= 0.0) and np.all(y <= 1.0)):
        fail("range", "y outside [0, 1]")
    order_x = np.argsort(x, axis=1, kind="stable")
    ys = np.take_along_axis(y, order_x, axis=1)
    if not np.all(np.diff(ys, axis=1) >= 0.0):
        fail("monotone", "larger x gave smaller y")
    perm = rng.permutation(x.shape[1])
    if not _close(sm(x[:, perm]), y[:, perm], 1e-15, 1e-300):
        fail("permutation", "column permutation changed the result")
    # exact shift invariance on a grid where x + c and x - max are exact
    xq = np.round(rng.normal(0.0, 5.0, size=(8, 64)) * 2.0 ** 16) / 2.0 ** 16
    yq = sm(xq)
    for c in (-3.0, 0.5, 1024.0):
        if not np.array_equal(sm(xq + c), yq):
            fail("shift", f"x + {c} changed the result")
    for cols in (1, 5, 64, 1000):
        yc = sm(np.full((2, cols), -2.75))
        if not np.all(yc == 1.0 / cols):
            fail("constant_row", f"cols={cols}")
    xd = np.full((3, 40), -1000.0)
    xd[np.arange(3), [0, 17, 39]] = 0.0
    yd = sm(xd)
    want = np.zeros_like(xd)
    want[np.arange(3), [0, 17, 39]] = 1.0
    if not np.array_equal(yd, want):
        fail("one_hot", "dominant entry is not exactly one-hot")
    xm = rng.normal(0.0, 1.0, size=(4, 32))
    xm[:, 5::3] = -np.inf
    ym = sm(xm)
    if not np.all(ym[:, 5::3] == 0.0) or not np.all(ym[:, :5] > 0.0):
        fail("masked", "-inf entries are not exactly 0")
    if not np.all(sm(rng.normal(0.0, 50.0, size=(5, 1))) == 1.0):
        fail("one_column", "C == 1 did not give 1")
    xs = np.array([[np.nan, 1.0, 2.0], [np.inf, 1.0, 2.0], [-np.inf] * 3, [0.0, 1.0, 2.0]])
    ys_ = sm(xs)
    if not (np.all(np.isnan(ys_[:3])) and not np.any(np.isnan(ys_[3]))):
        fail("special_rows", f"got {ys_.tolist()}")
    xt = rng.normal(0.0, 2.0, size=(37, 50))
    y1 = sm(xt, threads=1)
    for th in (2, 3, 8):
        if not np.array_equal(sm(xt, threads=th), y1):
            fail("threads", f"threads={th} differs from threads=1")

    # --- independent library implementations ----------------------------
    import scipy.special
    import torch
    xl = rng.normal(0.0, 4.0, size=(32, 300))
    yl = sm(xl)
    # The libraries sum in other orders and use other exp kernels: agreement
    # to 1e-14 relative (about 45 fp64 ulps) is what rounding allows here.
    if not _close(yl, scipy.special.softmax(xl, axis=-1), 1e-14):
        fail("scipy", "differs from scipy.special.softmax by > 1e-14 relative")
    yt = torch.softmax(torch.from_numpy(xl), dim=-1).numpy()
    if not _close(yl, yt, 1e-14):
        fail("torch", "differs from torch.softmax(float64) by > 1e-14 relative")

    # --- orientation -------------------------------------------------------
    xo = rng.normal(0.0, 1.0, size=(3, 11))
    yo = sm(xo)
    if not np.allclose(yo.sum(axis=1), 1.0, rtol=0, atol=1e-14):
        fail("orientation", "rows of a 3 x 11 input do not sum to 1")
    return fails


# ---------------------------------------------------------------------------
# Scaled, causally masked rows: y = softmax(scale * x + mask), mask(r, c) =
# -inf where period > 0 and c > (r mod period) + offset.

def brute_force_scaled_causal(x, scale, period, offset):
    """50-digit brute force of the masked, scaled definition, written from the
    definition: kept columns K(r) = {c : period == 0 or c <= r mod period +
    offset}; y_i = 1 / sum_{j in K} exp(scale (x_j - x_i)) for i in K, 0
    otherwise; NaN for a row with no kept column."""
    import mpmath
    mpmath.mp.dps = 50
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    for r in range(x.shape[0]):
        kept = [c for c in range(x.shape[1])
                if period == 0 or c <= (r % period) + offset]
        if not kept:
            out[r, :] = np.nan
            continue
        for i in kept:
            tot = mpmath.mpf(0)
            for j in kept:
                tot += mpmath.exp(mpmath.mpf(scale) * (mpmath.mpf(float(x[r, j])) -
                                                       mpmath.mpf(float(x[r, i]))))
            out[r, i] = float(1 / tot)
    return out


def run_fused_pins(smf, sm_plain) -> list:
    """smf(x, scale, period, offset, threads=1) -> y; sm_plain = the pinned
    plain oracle, used only for the masked-data identity."""
    fails = []

    def fail(name, msg):
        fails.append(f"{name}: {msg}")

    rng = np.random.default_rng(99)
    for scale in (0.125, 1.0, -0.5, 3.0):
        for period, offset in ((0, 0), (1, 0), (3, 0), (5, 2), (4, -1), (7, 3)):
            x = rng.normal(0.0, 4.0, size=(9, 11))
            y = np.asarray(smf(x, scale, period, offset))
            v = brute_force_scaled_causal(x, scale, period, offset)
            gap = np.abs(scale) * np.abs(x - np.nanmax(x, axis=1, keepdims=True))
            rel = (16.0 + 4.0 * gap + x.shape[1]) * 2.0 ** -53
            ok = y.shape == v.shape and np.array_equal(np.isnan(y), np.isnan(v))
            if ok:
                f = ~np.isnan(v)
                ok = bool(np.all(np.abs(y[f] - v[f]) <= rel[f] * np.abs(v[f]) + 2.0 ** -1070))
            if not ok:
                fail("fused_brute_force", f"scale={scale} period={period} offset={offset}")

    # identity: scale 1 and the mask written into the data as -inf equal the
    # plain definition, bit for bit (same arithmetic)
    x = rng.normal(0.0, 2.0, size=(12, 17))
    for period, offset in ((4, 0), (12, 5), (3, -1)):
        xm = x.copy()
        for r in range(x.shape[0]):
            xm[r, (r % period) + offset + 1:] = -np.inf
            if (r % period) + offset < 0:
                xm[r, :] = -np.inf
        if not np.array_equal(np.asarray(smf(x, 1.0, period, offset)), np.asarray(sm_plain(xm)),
                              equal_nan=True):
            fail("masked_data_identity", f"period={period} offset={offset}")

    # power-of-two scale: scale * x is exact, so scale=4 on x equals scale=1 on 4x
    xq = np.round(rng.normal(0.0, 3.0, size=(6, 20)) * 256.0) / 256.0
    if not np.array_equal(np.asarray(smf(xq, 4.0, 6, 0)), np.asarray(smf(4.0 * xq, 1.0, 6, 0)),
                          equal_nan=True):
        fail("pow2_scale", "scale 4 differs from pre-scaled data")

    # causal structure: query 0 with offset 0 keeps column 0 only -> one-hot;
    # masked entries are exactly 0; a row with nothing kept is NaN
    x = rng.normal(0.0, 1.0, size=(8, 8))
    y = np.asarray(smf(x, 0.7, 4, 0))
    if not (y[0, 0] == 1.0 and np.all(y[0, 1:] == 0.0) and y[4, 0] == 1.0):
        fail("one_hot_query0", f"row 0 {y[0].tolist()}")
    for r in range(8):
        if not np.all(y[r, (r % 4) + 1:] == 0.0):
            fail("masked_zero", f"row {r}")
    yn = np.asarray(smf(x, 1.0, 4, -1))
    if not (np.all(np.isnan(yn[0])) and np.all(np.isnan(yn[4])) and not np.isnan(yn[1, 0])):
        fail("empty_row_nan", "query 0 with offset -1 should keep nothing")
    return fails


# ---------------------------------------------------------------------------
# Log-softmax: y_j = x_j - log(sum_k exp(x_k)).

def brute_force_log_softmax(x):
    """50-digit y_i = -log(sum_j exp(x_j - x_i)): a different formula (no max,
    no separate log of a sum of shifted terms)."""
    import mpmath
    mpmath.mp.dps = 50
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    for r in range(x.shape[0]):
        row = [mpmath.mpf(float(v)) for v in x[r]]
        for i, xi in enumerate(row):
            if mpmath.isinf(xi) and xi < 0:
                out[r, i] = -np.inf
                continue
            tot = mpmath.mpf(0)
            for xj in row:
                if not (mpmath.isinf(xj) and xj < 0):
                    tot += mpmath.exp(xj - xi)
            out[r, i] = float(-mpmath.log(tot))
    return out


def run_log_pins(lsm) -> list:
    fails = []

    def fail(name, msg):
        fails.append(f"{name}: {msg}")

    for x in brute_force_inputs():
        y = np.asarray(lsm(x))
        v = brute_force_log_softmax(x)
        fin = np.isfinite(v)
        m = np.max(np.where(np.isneginf(x), -np.inf, x), axis=1, keepdims=True)
        tol = (8.0 + x.shape[1]) * 2.0 ** -52 * (1.0 + np.abs(x) + np.abs(m) + np.abs(v))
        ok = y.shape == v.shape and np.array_equal(np.isneginf(y), np.isneginf(v)) and \
            np.array_equal(np.isnan(y), np.isnan(v))
        if ok:
            ok = bool(np.all(np.abs(y[fin] - v[fin]) <= tol[fin]))
        if not ok:
            fail("log_brute_force", f"shape {x.shape}")
    rng = np.random.default_rng(11)
    x = rng.normal(0.0, 3.0, size=(10, 57))
    y = np.asarray(lsm(x))
    if not np.all(np.abs(np.exp(y).sum(axis=1) - 1.0) <= 64 * 2.0 ** -52):
        fail("log_normalised", "sum exp(y) != 1")
    d_y = y[:, :, None] - y[:, None, :]
    d_x = x[:, :, None] - x[:, None, :]
    if not np.all(np.abs(d_y - d_x) <= 8 * 2.0 ** -52 * (np.abs(y).max() + np.abs(x).max())):
        fail("log_differences", "y_i - y_j != x_i - x_j")
    for cols in (1, 7, 1000):
        yc = np.asarray(lsm(np.zeros((2, cols))))
        if not np.all(yc == -np.log(float(cols))):
            fail("log_constant_row", f"cols={cols}")
    xd = np.full((2, 9), -1000.0)
    xd[:, 4] = 0.0
    yd = np.asarray(lsm(xd))
    if not (np.all(yd[:, 4] == 0.0) and np.all(yd[:, :4] == -1000.0)):
        fail("log_dominant", f"{yd[0].tolist()}")
    xs = np.array([[np.nan, 1.0], [np.inf, 1.0], [-np.inf, -np.inf], [-np.inf, 2.0]])
    ys = np.asarray(lsm(xs))
    if not (np.all(np.isnan(ys[:3])) and ys[3, 0] == -np.inf and ys[3, 1] == 0.0):
        fail("log_special_rows", f"{ys.tolist()}")
    return fails


# ---------------------------------------------------------------------------
# Softmax backward: dx = y * (dy - sum(y * dy)).

def brute_force_backward(y, dy):
    """50-digit product of the softmax Jacobian J = diag(y) - y y^T with dy,
    formed as a full matrix (the oracle uses a dot product instead)."""
    import mpmath
    mpmath.mp.dps = 50
    out = np.empty_like(np.asarray(y, dtype=np.float64))
    for r in range(y.shape[0]):
        yr = [mpmath.mpf(float(v)) for v in y[r]]
        dr = [mpmath.mpf(float(v)) for v in dy[r]]
        n = len(yr)
        for i in range(n):
            acc = mpmath.mpf(0)
            for j in range(n):
                jac = yr[i] * ((1 if i == j else 0) - yr[j])
                acc += jac * dr[j]
            out[r, i] = float(acc)
    return out


def run_backward_pins(bwd, sm) -> list:
    """bwd(y, dy) -> dx; sm = the pinned softmax oracle (for finite
    differences and for probability rows)."""
    fails = []

    def fail(name, msg):
        fails.append(f"{name}: {msg}")

    rng = np.random.default_rng(5)
    for cols in (1, 2, 5, 16, 33):
        y = np.asarray(sm(rng.normal(0.0, 2.0, size=(4, cols))))
        dy = rng.normal(0.0, 1.0, size=(4, cols))
        dx = np.asarray(bwd(y, dy))
        v = brute_force_backward(y, dy)
        tol = (16.0 + cols) * 2.0 ** -52 * (np.abs(y) * (np.abs(dy) + np.sum(np.abs(y * dy), axis=1,
                                                                            keepdims=True)) + 1e-300)
        if not (dx.shape == v.shape and np.all(np.abs(dx - v) <= tol)):
            fail("backward_brute_force", f"cols={cols}")
    # the gradient of L(x) = sum(dy * softmax(x)) by central differences
    x = rng.normal(0.0, 1.5, size=(3, 12))
    dy = rng.normal(0.0, 1.0, size=(3, 12))
    y = np.asarray(sm(x))
    dx = np.asarray(bwd(y, dy))
    h = 1e-6
    fd = np.empty_like(x)
    for j in range(x.shape[1]):
        xp, xm = x.copy(), x.copy()
        xp[:, j] += h
        xm[:, j] -= h
        fd[:, j] = ((np.asarray(sm(xp)) * dy).sum(1) - (np.asarray(sm(xm)) * dy).sum(1)) / (2 * h)
    if not np.all(np.abs(fd - dx) <= 1e-8):
        fail("backward_finite_difference", f"max {np.max(np.abs(fd - dx)):.2e}")
    # rows of a probability vector: sum(dx) = dot * (1 - sum(y)) = 0; adding a
    # constant to dy changes nothing
    y = np.asarray(sm(rng.normal(0.0, 3.0, size=(6, 50))))
    dy = rng.normal(0.0, 1.0, size=(6, 50))
    dx = np.asarray(bwd(y, dy))
    if not np.all(np.abs(dx.sum(1)) <= 1e-14):
        fail("backward_sum_zero", f"{np.abs(dx.sum(1)).max():.2e}")
    if not np.allclose(np.asarray(bwd(y, dy + 3.0)), dx, rtol=0, atol=1e-14):
        fail("backward_shift", "dy + c changed dx")
    return fails


# ---------------------------------------------------------------------------
# MoE group score: per group of G scores, the sum of the two largest values.

def _f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def _bf16_rne(x32):
    """fp32 values -> nearest bf16 (ties to even), as fp64; NaN kept."""
    a = np.asarray(x32, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000).astype(np.uint32)
    out = r.view(np.float32).astype(np.float64)
    return np.where(np.isnan(a), np.nan, out)


def brute_force_group_pairs(scores, group, out_dtype="f32"):
    """The paper's identity written out: max over i != j of v_i + v_j (every
    ordered pair, the diagonal excluded), the exact double sum of two stored
    values rounded once to float, then to bf16 if asked.  NaN in a group -> NaN."""
    s = np.asarray(scores, dtype=np.float64)
    t, e = s.shape
    v = s.reshape(t, e // group, group)
    with np.errstate(invalid="ignore"):
        pair = v[..., :, None] + v[..., None, :]
    eye = np.eye(group, dtype=bool)
    pair = np.where(eye, -np.inf, pair)
    has_nan = np.isnan(v).any(axis=-1)
    with np.errstate(invalid="ignore"):
        best = np.where(np.isnan(pair), -np.inf, pair).max(axis=(-1, -2))
    # a pair sum that is NaN without a NaN input is +inf + -inf: keep it only
    # when no larger pair exists
    inf_nan = np.isnan(pair).any(axis=(-1, -2)) & ~has_nan & (best == -np.inf)
    best = np.where(has_nan | inf_nan, np.nan, best)
    r = _f32(best)
    return _bf16_rne(r) if out_dtype == "bf16" else r


def _same(a, b):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    return a.shape == b.shape and np.array_equal(np.isnan(a), np.isnan(b)) and \
        bool(np.all((a == b) | np.isnan(a)))


def run_moe_pins(fn) -> list:
    """fn(scores, group, out_dtype) -> group scores (fp64 array)."""
    import torch
    fails = []

    def fail(name, msg):
        fails.append(f"{name}: {msg}")

    rng = np.random.default_rng(21)
    for group in (2, 4, 8, 32, 64):
        # bf16-valued scores: ties are frequent, as with low-precision routing scores
        x = rng.normal(size=(40, 4 * group))
        xb = torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
        for dt in ("f32", "bf16"):
            if not _same(fn(xb, group, dt), brute_force_group_pairs(xb, group, dt)):
                fail("pairwise_identity", f"group={group} {dt}")
        tk = torch.topk(torch.tensor(xb).view(40, 4, group), 2, dim=-1).values.sum(-1)
        if not _same(fn(xb, group, "f32"), _f32(tk.view(40, 4).numpy())):
            fail("torch_topk", f"group={group}")
    # sums that are not floats: rounded once to float
    x = np.array([[1.0, 2.0 ** -30, -5.0, 0.0]])
    if not _same(fn(x, 4, "f32"), [[1.0]]):
        fail("float_rounding", f"{fn(x, 4, 'f32')}")
    x = np.array([[1.0, 1.0 + 2.0 ** -23, -1.0, 3.0 * 2.0 ** -25]])
    if not _same(fn(x, 4, "f32"), _f32([[2.0 + 2.0 ** -23]])):
        fail("float_rounding_2", f"{fn(x, 4, 'f32')}")
    # ties: a maximum that occurs twice counts twice (value masking would
    # give 5 + 1)
    x = np.array([[5.0, 1.0, 5.0, -2.0, 0.5, 1.0, 1.0, 0.0]])
    if not _same(fn(x, 8, "f32"), [[10.0]]):
        fail("tied_max", f"{fn(x, 8, 'f32')}")
    if not _same(fn(np.full((1, 32), -0.75), 32, "f32"), [[-1.5]]):
        fail("constant_group", "")
    x = np.array([[3.0, 1.0, 2.0, 2.0, -9.0, 7.0, 7.0, 7.0]])
    if not _same(fn(x, 4, "f32"), [[5.0, 14.0]]):
        fail("two_groups", f"{fn(x, 4, 'f32')}")
    # special values
    x = np.array([[np.nan, 1.0, 2.0, 3.0], [1.0, 2.0, np.nan, 3.0],
                  [np.inf, -np.inf, -np.inf, -np.inf],
                  [np.inf, np.inf, 0.0, 1.0], [-np.inf, -np.inf, -np.inf, -np.inf],
                  [-np.inf, 4.0, -np.inf, -np.inf], [np.inf, 1.0, -np.inf, 2.0]])
    want = [[np.nan], [np.nan], [np.nan], [np.inf], [-np.inf], [-np.inf], [np.inf]]
    if not _same(fn(x, 4, "f32"), want):
        fail("special_values", f"{fn(x, 4, 'f32').ravel().tolist()}")
    # bf16 output rounds the float sum to nearest, ties to even
    x = np.array([[1.0, 2.0 ** -8, 0.0, -1.0], [1.0, 3.0 * 2.0 ** -8, 0.0, -1.0],
                  [1.0, 2.0 ** -9, 0.0, -1.0]])
    if not _same(fn(x, 4, "bf16"), [[1.0], [1.0 + 2.0 ** -6], [1.0]]):
        fail("bf16_ties_to_even", f"{fn(x, 4, 'bf16').ravel().tolist()}")
    # order inside a group does not matter
    x = rng.normal(size=(16, 32))
    p = rng.permutation(32)
    if not _same(fn(x, 32, "f32"), fn(x[:, p], 32, "f32")):
        fail("permutation", "")
    return fails
