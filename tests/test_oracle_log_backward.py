"""The log-softmax and softmax-backward oracles against their pins, and
planted mistakes in them (no GPU)."""
import os

import pytest

import oracle
from oracle_pins import run_backward_pins, run_log_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "softmax_f64.c")


def _log(lib):
    return lambda x, threads=1: oracle.log_softmax_f64(x, threads=threads, lib=lib)


def _bwd(lib):
    return lambda y, dy: oracle.softmax_backward_f64(y, dy, lib=lib)


def _sm(lib):
    return lambda x, threads=1: oracle.softmax_f64(x, threads=threads, lib=lib)


def test_log_softmax_oracle_passes_every_pin():
    assert run_log_pins(_log(oracle.load())) == []


def test_backward_oracle_passes_every_pin():
    lib = oracle.load()
    assert run_backward_pins(_bwd(lib), _sm(lib)) == []


def test_backward_matches_torch_autograd():
    import numpy as np
    import torch
    rng = np.random.default_rng(1)
    x = rng.normal(0.0, 2.0, size=(7, 31))
    dy = rng.normal(0.0, 1.0, size=(7, 31))
    xt = torch.from_numpy(x).requires_grad_()
    torch.softmax(xt, -1).backward(torch.from_numpy(dy))
    dx = oracle.softmax_backward_f64(oracle.softmax_f64(x), dy)
    assert np.abs(dx - xt.grad.numpy()).max() <= 1e-15


LOG_MUTANTS = {
    "log_dropped": ("double lse = m + log(sum_e);", "double lse = m + sum_e - 1.0;"),
    "log_no_max": ("double lse = m + log(sum_e);", "double lse = log(sum_e);"),
    "log_sign": ("y[j] = x[j] - lse;", "y[j] = lse - x[j];"),
    "log_sum_unshifted": ("sum_e += exp(x[j] - m);", "sum_e += exp(x[j]);"),
    "log_min_not_max": ("m = fmax(m, x[j]);", "m = fmin(m, x[j]);"),
    "log_lse_halved": ("y[j] = x[j] - lse;", "y[j] = x[j] - 0.5 * lse;"),
}
BACKWARD_MUTANTS = {
    "bwd_dot_without_y": ("dot += yv[k] * dy[k];", "dot += dy[k];"),
    "bwd_sign": ("dx[j] = yv[j] * (dy[j] - dot);", "dx[j] = yv[j] * (dot - dy[j]);"),
    "bwd_missing_y": ("dx[j] = yv[j] * (dy[j] - dot);", "dx[j] = (dy[j] - dot);"),
    "bwd_dot_squared": ("dot += yv[k] * dy[k];", "dot += yv[k] * yv[k] * dy[k];"),
}


def _mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    return oracle.load(oracle.build(str(path), str(tmp_path / f"lib{name}.so")))


@pytest.mark.parametrize("name", sorted(LOG_MUTANTS))
def test_log_mutant_fails_a_pin(name, tmp_path):
    lib = _mutant(tmp_path, name, *LOG_MUTANTS[name])
    assert run_log_pins(_log(lib)), f"mutant {name} passed"


@pytest.mark.parametrize("name", sorted(BACKWARD_MUTANTS))
def test_backward_mutant_fails_a_pin(name, tmp_path):
    lib = _mutant(tmp_path, name, *BACKWARD_MUTANTS[name])
    assert run_backward_pins(_bwd(lib), _sm(oracle.load())), f"mutant {name} passed"
