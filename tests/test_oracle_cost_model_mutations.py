"""Plausible slips planted in a copy of the cost-model oracle must each fail a pin."""
import importlib.util
import os
import sys

import pytest

from oracle import cost_model
from tests import test_oracle_cost_model as pins

MUTATIONS = {
    "partial_w_off_by_one": ('partial = base * hh * (N["w"] - T["w"])', 'partial = base * hh * (N["w"] - T["w"] + 1)'),
    "halo_off_by_one": ('(T["h"] + T["r"] - 1) * (T["w"] + T["s"] - 1)', '(T["h"] + T["r"]) * (T["w"] + T["s"] - 1)'),
    "strict_outer_in_case1": ("if pos[j] >= ra), start", "if pos[j] > ra), start"),
    "case2_includes_ra": ("if pos[j] > ra), start=Fraction(1))\n        base", "if pos[j] >= ra), start=Fraction(1))\n        base"),
    "out_counted_once": ("def data_volume(perm, N, T, out_factor=2)", "def data_volume(perm, N, T, out_factor=1)"),
    "ker_missing_c": ('return T["k"] * T["c"] * T["r"] * T["s"]', 'return T["k"] * T["r"] * T["s"]'),
    "k_present_in_in": ('"In": frozenset("nchrws")', '"In": frozenset("nchrwsk")'),
    "r_not_sliding": ('SLIDING = frozenset("whsr")', 'SLIDING = frozenset("whs")'),
    "capacity_strict": ("for a in ARRAYS) <= capacity", "for a in ARRAYS) < capacity"),
    "capacity_drops_out": ("sum(footprint(a, T) for a in ARRAYS)", "sum(footprint(a, T) for a in ARRAYS[:2])"),
    "minmax_takes_min": ("return max(Fraction(d) / Fraction(bw)", "return min(Fraction(d) / Fraction(bw)"),
    "minmax_multiplies_bw": ("Fraction(d) / Fraction(bw) for d, bw", "Fraction(d) * Fraction(bw) for d, bw"),
    "multilevel_no_outer_reps": ("out.append(reps * data_volume(", "out.append(data_volume("),
}

PIN_FUNCS = (
    lambda: pins.test_matmul_eq3(),
    lambda: [pins.test_class_closed_forms(ci) for ci in range(8)],
    lambda: pins.test_full_tiles_give_compulsory_volume(),
    lambda: pins.test_rule_matches_previous_tile_cache_simulation(),
    lambda: pins.test_r_a_worked_example(),
    lambda: pins.test_capacity_eq4_hand_computed(),
    lambda: pins.test_minmax_objective_hand_computed(),
    lambda: pins.test_multilevel_counts_outer_tiles(),
)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_cost_model_pins_catch_planted_mistake(name, monkeypatch):
    src = open(cost_model.__file__).read()
    old, new = MUTATIONS[name]
    assert old in src, f"mutation anchor not found: {old!r}"
    spec = importlib.util.spec_from_loader("mutant_cost_model", loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src.replace(old, new, 1), "mutant_cost_model", "exec"), mod.__dict__)
    monkeypatch.setattr(pins, "cm", mod)
    failed = 0
    for f in PIN_FUNCS:
        try:
            f()
        except (AssertionError, ValueError, KeyError, ZeroDivisionError):
            failed += 1
    assert failed, f"mutation {name} passed every pin"
