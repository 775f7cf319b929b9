"""The scaled, causally masked oracle against its pins, and planted mistakes
in it (no GPU)."""
import os

import pytest

import oracle
from oracle_pins import run_fused_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "softmax_f64.c")


def _fused(lib):
    return lambda x, s, p, o, threads=1: oracle.softmax_scaled_causal_f64(
        x, s, p, o, threads=threads, lib=lib)


def _plain(lib):
    return lambda x, threads=1: oracle.softmax_f64(x, threads=threads, lib=lib)


def test_fused_oracle_passes_every_pin():
    lib = oracle.load()
    assert run_fused_pins(_fused(lib), _plain(lib)) == []


def test_sampled_rows_keep_their_mask():
    import numpy as np
    x = np.random.default_rng(3).normal(0.0, 2.0, size=(10, 12))
    full = oracle.softmax_scaled_causal_f64(x, 0.3, 4, 1)
    part = oracle.softmax_scaled_causal_f64(x[5:9], 0.3, 4, 1, row0=5)
    assert np.array_equal(full[5:9], part, equal_nan=True)


MUTANTS = {
    "mask_off_by_one": ("j > (r % period) + offset;", "j >= (r % period) + offset;"),
    "scale_magnitude_dropped": ("t[j] = masked ? -INFINITY : scale * x[j];",
                                "t[j] = masked ? -INFINITY : (scale > 0.0 ? x[j] : -x[j]);"),
    "divide_by_scale": ("t[j] = masked ? -INFINITY : scale * x[j];",
                        "t[j] = masked ? -INFINITY : x[j] / scale;"),
    "query_not_reduced": ("j > (r % period) + offset;", "j > r + offset;"),
    "offset_sign": ("j > (r % period) + offset;", "j > (r % period) - offset;"),
    "mask_ignored": ("int masked = period > 0 && j > (r % period) + offset;",
                     "int masked = period < 0 && j > (r % period) + offset;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_fused_mutant_fails_a_pin(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = oracle.load(oracle.build(str(path), str(tmp_path / f"lib{name}.so")))
    assert run_fused_pins(_fused(lib), _plain(oracle.load())), f"mutant {name} passed"
