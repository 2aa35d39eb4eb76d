"""The layer oracle's pins must catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of ``oracle/layer.py``, loads the copy
as a module, and runs the pins of ``test_oracle_layer.py`` against it: at least
one pin must fail for every mutant.
"""
import os
import types

import pytest

from tests import test_oracle_layer as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "layer.py")

MUTANTS = {
    "sine with the wrong sign": ("first * c - second * s", "first * c + second * s"),
    "second element rotated the other way": ("first * s + second * c", "-first * s + second * c"),
    "pairs taken as the two halves": (
        "first, second = x[..., 0::2], x[..., 1::2]",
        "first, second = x[..., :x.shape[-1] // 2], x[..., x.shape[-1] // 2:]"),
    "frequency exponent 2 i / n": ("-np.arange(n, dtype=np.float64) / n",
                                   "-2.0 * np.arange(n, dtype=np.float64) / n"),
    "frequency exponent i / (n - 1)": ("-np.arange(n, dtype=np.float64) / n",
                                       "-np.arange(n, dtype=np.float64) / max(n - 1, 1)"),
    "grid read column-major": ("for a in range(len(grid) - 1, -1, -1):", "for a in range(len(grid)):"),
    "every group turns with the first axis": ("coords[:, a:a + 1].astype", "coords[:, 0:1].astype"),
    "values rotated too": ("k = rope(k, angles)\n    S = q.shape[0]",
                           "k = rope(k, angles)\n    v = rope(v, angles)\n    S = q.shape[0]"),
    "keys not rotated": ("k = rope(k, angles)\n    S = q.shape[0]", "S = q.shape[0]"),
    "projection row head-major instead of q/k/v-major": (
        "t = qkv.reshape(S, 3, H, d)", "t = qkv.reshape(S, H, 3, d).transpose(0, 2, 1, 3)"),
    "heads concatenated in reverse": ("scale, rows) for h in range(H)], axis=1)",
                                      "scale, rows) for h in range(H)][::-1], axis=1)"),
}

PINS = [
    pins.test_grid_coords_brute_force,
    pins.test_worked_rotation_by_one_radian,
    pins.test_rotation_is_complex_multiplication,
    pins.test_norm_of_every_pair_is_preserved_and_position_zero_is_identity,
    lambda: pins.test_scores_depend_only_on_the_offset((40,), (8,)),
    lambda: pins.test_scores_depend_only_on_the_offset((4, 5, 6), (3, 3, 2)),
    pins.test_frequency_schedule_is_geometric_from_one_to_one_over_base,
    pins.test_each_axis_turns_only_its_own_group,
    pins.test_linear_brute_force,
    pins.test_split_layout_is_q_heads_then_k_heads_then_v_heads,
    pins.test_rope_pack_is_rope_then_the_pack_index_formula,
    pins.test_layer_reduces_to_attention_with_identity_weights_and_no_rotation,
    lambda: pins.test_layer_matches_pytorch_float64((48,), (4,), 2, 8, 20),
    lambda: pins.test_layer_matches_pytorch_float64((2, 4, 6), (2, 1, 1), 3, 8, 16),
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, monkeypatch):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert old in src, f"mutation site of {name!r} not found"
    mod = types.ModuleType("layer_mutant")
    exec(compile(src.replace(old, new), SRC, "exec"), mod.__dict__)
    monkeypatch.setattr(pins, "layer", mod)
    failed = 0
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            failed += 1
    assert failed >= 1, f"no pin caught {name!r}"


def test_unmutated_oracle_passes_every_pin():
    for pin in PINS:
        pin()
