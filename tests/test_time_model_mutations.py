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
    "partial round costs a full one": ("return full + length * (g0 + (1.0 - g0) * f)",
                                       "return full + length"),
    "partial round costs only its busy share": ("return full + length * (g0 + (1.0 - g0) * f)",
                                                "return full + length * f"),
    "lanes do not pool the rounds": ("attn = launch_rounds(sum(W), n_slots, g0, tail_ways(sum(W), n_slots, S, split))",
                                     "attn = sum(launch_rounds(w, n_slots, g0) for w in W)"),
    "lanes keep the pooled tail whole": ("attn = launch_rounds(sum(W), n_slots, g0, tail_ways(sum(W), n_slots, S, split))",
                                         "attn = launch_rounds(sum(W), n_slots, g0)"),
    "serial plan moves only the unpacks": ("copies = 4 * H ", "copies = H "),
    "one synchronisation per chunk": ("PIPELINED: 2 * C + 3", "PIPELINED: C + 3"),
    "fused launches always carry": ("if idle >= max(1, n_slots // 8):", "if True:"),
    "split tail keeps its full length": ("length = {1: 1.0, 2: 2.0 / 3.0, 3: 1.0 / 3.0}[ways]",
                                         "length = 1.0"),
    "split three ways where two fit": ("return 3 if 3 * rem <= n else", "return 3 if 2 * rem <= n else"),
    "drain once per plan": ("        attn += drain * C", "        attn += drain"),
}

PINS = [
    lambda: [pins.test_upper_bound_matches_printed_applicability_table(r, p)
             for r, p in ((0.35, 1.54), (0.20, 1.25), (0.10, 1.11))],
    pins.test_optimal_chunks_zeroes_the_derivative,
    pins.test_best_integer_is_next_to_the_real_optimum,
    pins.test_speedup_is_baseline_over_hcms_time,
    pins.test_one_chunk_pays_only_its_overhead,
    pins.test_fit_recovers_planted_parameters,
    pins.test_theory_validation_row_predicts_five_chunks,
    pins.test_round_identity,
    pins.test_one_gpu_model_reduces_to_the_paper_model,
    pins.test_worked_rounds_of_the_wan_p4_share,
    pins.test_worked_split_tails,
    pins.test_drain_adds_per_launch,
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
