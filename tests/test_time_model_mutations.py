"""The time-model oracle's pins must catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of ``oracle/time_model.py``, loads the
copy as a module, and runs the oracle pins of ``test_time_model.py`` against
it: at least one pin must fail for every mutant.
"""
import os
import types

import pytest

from tests import test_time_model as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "time_model.py")

MUTANTS = {
    "C* without the square root": ("math.sqrt(t_comm / beta)", "(t_comm / beta)"),
    "communication not divided by C": ("t0 + t_comm / C + t_attn + C * beta",
                                       "t0 + t_comm + t_attn + C * beta"),
    "overhead not multiplied by C": ("t0 + t_comm / C + t_attn + C * beta",
                                     "t0 + t_comm / C + t_attn + beta"),
    "speedup hides C instead of C - 1 chunks": ("rho * (C - 1) / C", "rho * C / (C + 1)"),
    "speedup overhead sign": ("+ C * beta_over_total", "- C * beta_over_total"),
    "integer optimum ignores the overhead": ("(t_comm / c + c * beta, c)", "(t_comm / c, c)"),
    "fit basis C instead of 1 / C": ("A = np.stack([np.ones_like(c), 1.0 / c, c], axis=1)",
                                     "A = np.stack([np.ones_like(c), c, c * c], axis=1)"),
}

PINS = [
    lambda: [pins.test_upper_bound_matches_printed_applicability_table(r, p)
             for r, p in ((0.35, 1.54), (0.20, 1.25), (0.10, 1.11))],
    pins.test_optimal_chunks_zeroes_the_derivative,
    pins.test_best_integer_is_next_to_the_real_optimum,
    pins.test_speedup_is_baseline_over_hcms_time,
    pins.test_one_chunk_pays_only_its_overhead,
    pins.test_fit_recovers_planted_parameters,
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, monkeypatch):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert old in src, f"mutation site of {name!r} not found"
    mod = types.ModuleType("time_model_mutant")
    exec(compile(src.replace(old, new), SRC, "exec"), mod.__dict__)
    monkeypatch.setattr(pins, "tm", mod)
    failed = 0
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ZeroDivisionError, ValueError):
            failed += 1
    assert failed >= 1, f"no pin caught {name!r}"


def test_unmutated_oracle_passes_every_pin():
    for pin in PINS:
        pin()
