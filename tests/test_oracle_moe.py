"""The MoE group-score oracle against its pins (the paper's pairwise identity
by brute force, torch.topk, closed forms, ties, special values, rounding), and
planted mistakes in it (no GPU)."""
import os

import pytest

import oracle
from oracle_pins import run_moe_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "moe_group_f64.c")


def _fn(lib):
    return lambda s, g, dt: oracle.moe_group_top2_f64(s, g, dt, lib=lib)


def test_moe_oracle_passes_every_pin():
    assert run_moe_pins(_fn(oracle.load_moe())) == []


def test_moe_oracle_rejects_bad_groups():
    import numpy as np
    with pytest.raises(ValueError):
        oracle.moe_group_top2_f64(np.zeros((2, 10)), 4)
    with pytest.raises(ValueError):
        oracle.moe_group_top2_f64(np.zeros((2, 10)), 1)


MUTANTS = {
    # the paper's failing variant: masking every value equal to the maximum
    "value_masking": ("if (i != p && v[i] > t2)", "if (v[i] != v[p] && v[i] > t2)"),
    "top1_twice": ("float s = (float)(v[p] + t2);", "float s = (float)(v[p] + v[p]);"),
    "min_not_max": ("if (v[i] > v[p])", "if (v[i] < v[p])"),
    "last_value_skipped": ("    for (int64_t i = 0; i < g; ++i)\n        if (i != p",
                           "    for (int64_t i = 0; i < g - 1; ++i)\n        if (i != p"),
    "group_stride": ("out[k] = group_top2(scores + k * group, group, bf16_out);",
                     "out[k] = group_top2(scores + k * (group - 1), group, bf16_out);"),
    "no_nan_rule": ("        if (isnan(v[i]))\n            return NAN;",
                    "        if (isnan(v[i]) && v[i] > 0)\n            return NAN;"),
    "sum_not_rounded": ("return bf16_out ? (double)round_to_bf16(s) : (double)s;",
                        "return bf16_out ? (double)round_to_bf16(s) : v[p] + t2;"),
    "bf16_ties_up": ("u += 0x7fffu + ((u >> 16) & 1u);", "u += 0x8000u;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_moe_mutant_fails_a_pin(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    lib = oracle.load_moe(oracle.build(str(path), str(tmp_path / f"lib{name}.so")))
    assert run_moe_pins(_fn(lib)), f"mutant {name} passed every pin"
