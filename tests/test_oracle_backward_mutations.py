"""The backward oracle's pins must catch plausible mistakes (CPU only): each
case plants one mistake in a copy of the oracle's C source and runs the pins
of ``test_oracle_backward.py`` against it."""
import pytest

from tests import test_oracle_backward as pins
from tests.test_oracle_mutations import _mutant_module

MUTANTS = {
    "softmax Jacobian without the row term": (
        "const double ds = exp(s[j] - mi) / li * (dp[j] - ci);",
        "const double ds = exp(s[j] - mi) / li * dp[j];"),
    "dq without the scale": ("o[t] += scale * ds * k[j * d + t];", "o[t] += ds * k[j * d + t];"),
    "dq sums values instead of keys": ("o[t] += scale * ds * k[j * d + t];",
                                       "o[t] += scale * ds * v[j * d + t];"),
    "dk from the transposed score": ("okk[t] += scale * ds * qi[t];", "okk[t] += scale * ds * kj[t];"),
    "dv weighted by ds instead of p": ("ov[t] += p * gi[t];", "ov[t] += ds * gi[t];"),
    "dp from keys instead of values": ("dg += gi[t] * v[j * d + t];", "dg += gi[t] * k[j * d + t];"),
    "row statistic not normalised": ("ci += exp(s[j] - mi) / li * dp[j];", "ci += exp(s[j] - mi) * dp[j];"),
    "pass 2 without the scale in p": ("const double p = exp(scale * dot - m[i]) / l[i];",
                                      "const double p = exp(dot - m[i]) / l[i];"),
}

PINS = [
    pins.test_matches_float64_autograd,
    pins.test_matches_central_differences_of_the_forward_oracle,
    pins.test_gradient_sums,
    pins.test_equal_keys_and_zero_scale,
    pins.test_single_key,
    pins.test_row_subsets_equal_full_rows,
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_backward_mutant(tmp_path, name):
    old, new = MUTANTS[name]
    mod = _mutant_module(tmp_path, name, old, new)
    caught = 0
    for pin in PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, FloatingPointError):
            caught += 1
    assert caught, f"no pin catches the mutant '{name}'"
