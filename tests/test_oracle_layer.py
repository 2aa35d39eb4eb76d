"""Pins of the layer oracle (projections and RoPE around the hot path), CPU only.

Each pin checks the oracle against something other than its own formulas: a
worked rotation with known values, complex multiplication, the relative-position
property RoPE is built for, brute-force loops, and PyTorch's float64 attention.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import layer


# ---------------------------------------------------------------------------
# Positions
# ---------------------------------------------------------------------------
def test_grid_coords_brute_force():
    grid = (2, 3, 4)
    want = [(f, r, c) for f in range(2) for r in range(3) for c in range(4)]
    assert layer.grid_coords(grid).tolist() == [list(w) for w in want]
    assert layer.grid_coords((7,)).ravel().tolist() == list(range(7))


# ---------------------------------------------------------------------------
# Rotation
# ---------------------------------------------------------------------------
def test_worked_rotation_by_one_radian():
    """One pair (d = 2) on a 1-D grid: pair 0 has frequency base^0 = 1, so the
    token at position 1 turns by exactly one radian: (1, 0) -> (cos 1, sin 1)
    and (0, 1) -> (-sin 1, cos 1)."""
    cos1, sin1 = 0.5403023058681398, 0.8414709848078965
    ang = layer.rope_angles((3,), (1,), base=10000.0)
    assert ang.ravel().tolist() == [0.0, 1.0, 2.0]
    x = np.array([[0.0, 0.0], [1.0, 0.0], [0.0, 0.0]])
    y = np.array([[0.0, 0.0], [0.0, 1.0], [0.0, 0.0]])
    assert layer.rope(x, ang)[1] == pytest.approx([cos1, sin1], abs=1e-15)
    assert layer.rope(y, ang)[1] == pytest.approx([-sin1, cos1], abs=1e-15)


def test_rotation_is_complex_multiplication():
    """Pair (x_2i, x_2i+1) as the complex number x_2i + i x_2i+1, multiplied by
    exp(i phi) (numpy's complex arithmetic, a separate formulation)."""
    rng = np.random.default_rng(1)
    S, H, d = 24, 3, 16
    x = rng.standard_normal((S, H, d))
    ang = layer.rope_angles((2, 3, 4), (3, 3, 2))
    z = (x[..., 0::2] + 1j * x[..., 1::2]) * np.exp(1j * ang)[:, None, :]
    want = np.stack([z.real, z.imag], axis=-1).reshape(S, H, d)
    assert np.abs(layer.rope(x, ang) - want).max() < 1e-13


def test_norm_of_every_pair_is_preserved_and_position_zero_is_identity():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((60, 2, 12))
    ang = layer.rope_angles((3, 4, 5), (2, 2, 2))
    r = layer.rope(x, ang)
    n0 = x[..., 0::2] ** 2 + x[..., 1::2] ** 2
    n1 = r[..., 0::2] ** 2 + r[..., 1::2] ** 2
    assert np.abs(n0 - n1).max() < 1e-12
    assert np.array_equal(r[0], x[0])          # token 0 sits at the origin


@pytest.mark.parametrize("grid,pairs", [((40,), (8,)), ((4, 5, 6), (3, 3, 2))])
def test_scores_depend_only_on_the_offset(grid, pairs):
    """RoPE's defining property: <R(q, t1), R(k, t2)> depends on the
    coordinates of t1 and t2 only through their difference on every axis."""
    rng = np.random.default_rng(3)
    d = 2 * sum(pairs)
    coords = layer.grid_coords(grid)
    ang = layer.rope_angles(grid, pairs)
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    S = coords.shape[0]
    Q = layer.rope(np.tile(q, (S, 1)), ang)
    K = layer.rope(np.tile(k, (S, 1)), ang)
    scores = {}
    for t1 in range(0, S, 7):
        for t2 in range(0, S, 5):
            key = tuple(coords[t1] - coords[t2])
            s = float(Q[t1] @ K[t2])
            if key in scores:
                assert s == pytest.approx(scores[key], abs=1e-11)
            scores[key] = s
    assert len(scores) > 10
    # and it does depend on the offset
    assert max(scores.values()) - min(scores.values()) > 1e-3


def test_frequency_schedule_is_geometric_from_one_to_one_over_base():
    """RoFormer's schedule over a group of n pairs: the first pair turns at one
    radian per unit of position and each next pair slower by the same ratio r,
    with r^n = 1 / base."""
    base = 500.0
    for pairs in ((6,), (4, 3, 5)):
        grid = tuple(2 for _ in pairs)
        ang = layer.rope_angles(grid, pairs, base=base)
        coords = layer.grid_coords(grid)
        start = 0
        for a, n in enumerate(pairs):
            t = int(np.flatnonzero((coords[:, a] == 1) & (coords.sum(axis=1) == 1))[0])
            g = ang[t, start:start + n]
            assert g[0] == pytest.approx(1.0, abs=1e-15)
            if n > 1:
                r = g[1:] / g[:-1]
                assert np.allclose(r, r[0], rtol=1e-12)
                assert r[0] ** n == pytest.approx(1.0 / base, rel=1e-12)
            assert np.all(np.delete(ang[t], np.s_[start:start + n]) == 0.0)
            start += n


def test_each_axis_turns_only_its_own_group():
    grid, pairs = (3, 4, 5), (2, 3, 1)
    coords = layer.grid_coords(grid)
    ang = layer.rope_angles(grid, pairs)
    bounds = np.cumsum((0,) + pairs)
    for t1 in range(coords.shape[0]):
        for t2 in range(coords.shape[0]):
            for a in range(3):
                same = coords[t1, a] == coords[t2, a]
                g1 = ang[t1, bounds[a]:bounds[a + 1]]
                g2 = ang[t2, bounds[a]:bounds[a + 1]]
                assert np.array_equal(g1, g2) == same


# ---------------------------------------------------------------------------
# Projections and the split of the projection output
# ---------------------------------------------------------------------------
def test_linear_brute_force():
    rng = np.random.default_rng(4)
    x, w = rng.standard_normal((5, 7)), rng.standard_normal((7, 3))
    want = [[sum(x[i, k] * w[k, j] for k in range(7)) for j in range(3)] for i in range(5)]
    assert np.abs(layer.linear(x, w) - np.array(want)).max() < 1e-13


def test_split_layout_is_q_heads_then_k_heads_then_v_heads():
    S, H, d = 3, 2, 4
    row = np.concatenate([np.full(d, 100 * which + 10 * h) for which in range(3) for h in range(H)])
    qkv = np.stack([row + t for t in range(S)])
    q, k, v = layer.split_qkv(qkv, H, d)
    for t in range(S):
        for h in range(H):
            assert np.all(q[t, h] == 10 * h + t)
            assert np.all(k[t, h] == 100 + 10 * h + t)
            assert np.all(v[t, h] == 200 + 10 * h + t)


def test_rope_pack_is_rope_then_the_pack_index_formula():
    rng = np.random.default_rng(5)
    S, H, d, P = 24, 4, 8, 4
    qkv = rng.standard_normal((S, 3 * H * d))
    ang = layer.rope_angles((2, 3, 4), (2, 1, 1))
    q, k, v = layer.split_qkv(qkv, H, d)
    qr, kr = layer.rope(q, ang), layer.rope(k, ang)
    for h0, hc in ((0, 4), (1, 2), (3, 1)):
        gq, gk, gv = layer.rope_pack(qkv, ang, H, d, h0, hc)
        assert np.array_equal(gq, oracle.pack(np.ascontiguousarray(qr), P, h0, hc))
        assert np.array_equal(gk, oracle.pack(np.ascontiguousarray(kr), P, h0, hc))
        assert np.array_equal(gv, oracle.pack(np.ascontiguousarray(v), P, h0, hc))


# ---------------------------------------------------------------------------
# The layer
# ---------------------------------------------------------------------------
def test_layer_reduces_to_attention_with_identity_weights_and_no_rotation():
    rng = np.random.default_rng(6)
    S, H, d = 40, 2, 8
    x = rng.standard_normal((S, H * d))
    eye = np.eye(H * d)
    w_qkv = np.concatenate([eye, eye, eye], axis=1)
    y = layer.layer_forward(x, w_qkv, eye, np.zeros((S, d // 2)), H, d, 0.3, oracle.attention_head)
    xs = x.reshape(S, H, d)
    for h in range(H):
        o = oracle.attention_head(xs[:, h], xs[:, h], xs[:, h], 0.3)
        assert np.abs(y[:, h * d:(h + 1) * d] - o).max() < 1e-13


def _torch_layer(x, w_qkv, w_o, ang, H, d, scale):
    """The same layer from PyTorch float64 primitives: matmul, complex
    rotation (torch.polar) and scaled_dot_product_attention."""
    x, w_qkv, w_o, ang = (torch.from_numpy(np.asarray(a, dtype=np.float64)) for a in (x, w_qkv, w_o, ang))
    S = x.shape[0]
    qkv = (x @ w_qkv).reshape(S, 3, H, d)
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]

    def turn(t):
        z = torch.view_as_complex(t.contiguous().reshape(S, H, d // 2, 2)) * rot
        return torch.view_as_real(z).reshape(S, H, d)

    q, k, v = turn(qkv[:, 0]), turn(qkv[:, 1]), qkv[:, 2]
    o = torch.nn.functional.scaled_dot_product_attention(
        q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1), scale=scale)
    return (o.transpose(0, 1).reshape(S, H * d) @ w_o).numpy()


@pytest.mark.parametrize("grid,pairs,H,d,D", [((48,), (4,), 2, 8, 20), ((2, 4, 6), (2, 1, 1), 3, 8, 16)])
def test_layer_matches_pytorch_float64(grid, pairs, H, d, D):
    rng = np.random.default_rng(7)
    S = int(np.prod(grid))
    x = rng.standard_normal((S, D))
    w_qkv = rng.standard_normal((D, 3 * H * d)) / math.sqrt(D)
    w_o = rng.standard_normal((H * d, D)) / math.sqrt(H * d)
    ang = layer.rope_angles(grid, pairs)
    y = layer.layer_forward(x, w_qkv, w_o, ang, H, d, d ** -0.5, oracle.attention_head)
    want = _torch_layer(x, w_qkv, w_o, ang, H, d, d ** -0.5)
    assert np.abs(y - want).max() < 1e-12
    rows = np.array([0, 5, S - 1])
    ys = layer.layer_forward(x, w_qkv, w_o, ang, H, d, d ** -0.5, oracle.attention_head, rows)
    assert np.abs(ys - y[rows]).max() < 1e-13
