"""The oracle's pins must catch plausible mistakes (CPU only).

Each case below plants one mistake in a copy of the oracle's C source, builds
it into a temporary library, and runs the pin tests of ``test_oracle.py``
against it.  At least one pin must fail for every mutant.
"""
import importlib.util
import os
import subprocess

import pytest

from tests import test_oracle as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "hcms_oracle.c")

MUTANTS = {
    "scale dropped": ("s[j] = scale * dot;", "s[j] = dot;"),
    "max not subtracted": ("const double w = exp(s[j] - m);", "const double w = exp(s[j]);"),
    "max subtracted with wrong sign": ("const double w = exp(s[j] - m);",
                                       "const double w = exp(m - s[j]);"),
    "no normalisation": ("for (int64_t t = 0; t < d; ++t) o[t] /= l;", ""),
    "values read from K": ("const double *vj = v + j * d;", "const double *vj = k + j * d;"),
    "key index is the query index": ("const double *kj = k + j * d;",
                                     "const double *kj = k + (i % S) * d;"),
    "value rows offset by one": ("const double *vj = v + j * d;",
                                 "const double *vj = v + ((j + 1) % S) * d;"),
    "exp2 instead of exp": ("const double w = exp(s[j] - m);",
                            "const double w = exp2(s[j] - m);"),
    "pack ignores h0": ("const int64_t from = ((p * Ss + s) * H + (h0 + j)) * d + e;",
                        "const int64_t from = ((p * Ss + s) * H + j) * d + e;"),
    "pack shards interleaved": ("const int64_t to = (j * S + (p * Ss + s)) * d + e;",
                                "const int64_t to = (j * S + (s * P + p)) * d + e;"),
    "unpack into wrong heads": ("const int64_t to = ((p * Ss + s) * H + (h0 + j)) * d + e;",
                                "const int64_t to = ((p * Ss + s) * H + (H - 1 - h0 - j)) * d + e;"),
}

PIN_TESTS = [
    lambda m: pins.test_two_key_worked_example(m),
    lambda m: pins.test_constant_values(m),
    lambda m: pins.test_equal_keys_and_zero_scale_give_mean(m),
    lambda m: pins.test_single_token(m),
    lambda m: pins.test_large_logits_do_not_overflow(m),
    lambda m: pins.test_planted_peak_selects_its_value_row(m),
    lambda m: pins.test_convex_hull(m),
    lambda m: pins.test_permutation_equivariance(m),
    lambda m: pins.test_matches_torch_sdpa_fp64(m, "tiny"),
    lambda m: [pins.test_pack_is_numpy_head_slice_transpose(m, *a) for a in
               [(4, 128, 4, 64, pins.np.float32), (3, 24, 7, 8, pins.np.uint16)]],
    lambda m: pins.test_pack_unpack_roundtrip_and_sentinels(m),
]


def _mutant_module(tmp_path, name, old, new):
    src = open(SRC).read()
    assert old in src, f"mutation site for '{name}' not found"
    mutated = src.replace(old, new, 1)
    c_path = tmp_path / "mutant.c"
    c_path.write_text(mutated)
    so_path = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                    "-o", str(so_path), str(c_path), "-lm"], check=True)
    spec = importlib.util.spec_from_file_location(
        "oracle_mutant", os.path.join(ROOT, "oracle", "__init__.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    mod._LIB_PATH = str(so_path)
    mod._lib = None
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(tmp_path, name):
    old, new = MUTANTS[name]
    mod = _mutant_module(tmp_path, name, old, new)
    caught = []
    for i, pin in enumerate(PIN_TESTS):
        try:
            pin(mod)
        except (AssertionError, ValueError, FloatingPointError):
            caught.append(i)
    assert caught, f"no pin catches the mutant '{name}'"
