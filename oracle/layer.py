"""Oracle for the attention layer around the hot path: QKV projection and rotary
position embedding before the split along heads, output projection after the
concatenation (Alg. 1, the main-stream steps; Sec. 2 lists the Ulysses forward
as projection, RoPE, input all-to-all, attention, output all-to-all, output
projection, and cites RoFormer for the position embedding).

TEST INFRASTRUCTURE ONLY.  The test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` are the only callers; the product path
never imports this module and this module never imports the product path.

Everything is float64 on the exact stored input values.  The paper names the
steps but prints no formula for them; the readings written out here are:

* Projection: ``qkv = X W_qkv`` with ``X`` ``[S][D]`` and ``W_qkv``
  ``[D][3 H d]``; a token's output row holds the H query heads, then the H key
  heads, then the H value heads, each ``d`` wide.  Output projection:
  ``Y = O W_o`` with ``O`` ``[S][H d]`` (the heads concatenated in head order,
  Alg. 1 Concat) and ``W_o`` ``[H d][D]``.  No bias terms.
* RoPE (RoFormer): pair ``i`` of a head vector is the element pair
  ``(2i, 2i+1)``; rotating it by the angle ``phi`` maps ``(x, y)`` to
  ``(x cos phi - y sin phi, x sin phi + y cos phi)``.  Queries and keys are
  rotated, values are not.
* Positions: the tokens of the sequence, in the global order
  ``t = p (S/P) + s``, fill a row-major grid ``G_0 x ... x G_{A-1}`` (for video
  latents: frames, rows, columns), so token ``t`` has one coordinate per axis.
  The ``d/2`` pairs form consecutive groups of ``n_0, ..., n_{A-1}`` pairs;
  group ``a`` turns with coordinate ``a``, and its pair ``i'`` has the
  frequency ``base^(-i'/n_a)``, RoFormer's geometric schedule over the group.
  A single axis is RoFormer's one-dimensional position.

The functions are pinned in ``tests/test_oracle_layer.py`` by a worked rotation,
the relative-position property of RoPE, a complex-multiplication formulation,
norm preservation, axis separation, brute-force products, and reductions of the
layer to plain attention.
"""
from __future__ import annotations

import numpy as np


# ---------------------------------------------------------------------------
# Positions and rotary angles
# ---------------------------------------------------------------------------
def grid_coords(grid) -> np.ndarray:
    """Coordinates ``[S][A]`` of the tokens ``t = 0 .. S-1`` on the row-major
    grid ``grid`` (``S`` = the product of the grid sizes); the last axis
    varies fastest."""
    grid = [int(g) for g in grid]
    if not grid or min(grid) < 1:
        raise ValueError("grid sizes must be >= 1")
    S = int(np.prod(grid))
    coords = np.empty((S, len(grid)), dtype=np.int64)
    rest = np.arange(S, dtype=np.int64)
    for a in range(len(grid) - 1, -1, -1):
        coords[:, a] = rest % grid[a]
        rest = rest // grid[a]
    return coords


def rope_angles(grid, axis_pairs, base: float = 10000.0) -> np.ndarray:
    """Rotation angle ``[S][d/2]`` of every pair of every token: the pairs of
    group ``a`` turn by ``coordinate_a * base^(-i'/n_a)``."""
    coords = grid_coords(grid)
    if len(axis_pairs) != coords.shape[1] or min(axis_pairs) < 1:
        raise ValueError("one positive pair count per grid axis")
    cols = []
    for a, n in enumerate(axis_pairs):
        freq = float(base) ** (-np.arange(n, dtype=np.float64) / n)
        cols.append(coords[:, a:a + 1].astype(np.float64) * freq[None, :])
    return np.concatenate(cols, axis=1)


def rope(x: np.ndarray, angles: np.ndarray) -> np.ndarray:
    """Rotate the pairs of ``x`` (``[S][d]`` or ``[S][H][d]``) by ``angles``
    (``[S][d/2]``, the same angles for every head of a token)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.asarray(angles, dtype=np.float64)
    if x.ndim == 3:
        a = a[:, None, :]
    if x.shape[-1] != 2 * a.shape[-1] or x.shape[0] != a.shape[0]:
        raise ValueError("angles must be [S][d/2] for x of [S](...)[d]")
    c, s = np.cos(a), np.sin(a)
    first, second = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = first * c - second * s
    out[..., 1::2] = first * s + second * c
    return out


# ---------------------------------------------------------------------------
# Projections
# ---------------------------------------------------------------------------
def linear(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """``x @ w`` in float64 (``x`` ``[M][K]``, ``w`` ``[K][N]``)."""
    return np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64)


def split_qkv(qkv: np.ndarray, H: int, d: int):
    """Views ``q``, ``k``, ``v`` ``[S][H][d]`` of a projection output
    ``[S][3 H d]``."""
    qkv = np.asarray(qkv)
    S = qkv.shape[0]
    if qkv.shape[1] != 3 * H * d:
        raise ValueError("projection output must be [S][3 H d]")
    t = qkv.reshape(S, 3, H, d)
    return t[:, 0], t[:, 1], t[:, 2]


def rope_pack(qkv: np.ndarray, angles: np.ndarray, H: int, d: int, h0: int, hc: int):
    """Head chunk ``[h0, h0 + hc)`` of the rotated queries and keys and of the
    values, head-major ``[hc][S][d]`` each: the split along heads of Alg. 1
    (and the local share of its input all-to-all) after RoPE."""
    q, k, v = split_qkv(qkv, H, d)
    sl = slice(h0, h0 + hc)
    qr = rope(q[:, sl], angles)
    kr = rope(k[:, sl], angles)
    return (np.ascontiguousarray(qr.transpose(1, 0, 2)),
            np.ascontiguousarray(kr.transpose(1, 0, 2)),
            np.ascontiguousarray(np.asarray(v[:, sl], dtype=np.float64).transpose(1, 0, 2)))


def layer_forward(x, w_qkv, w_o, angles, H: int, d: int, scale: float, attention_head,
                  rows=None) -> np.ndarray:
    """``Y`` ``[len(rows)][D]`` for the token rows ``rows`` (default all):
    projection, RoPE on Q and K, attention of every head (``attention_head``,
    the per-head attention oracle, called as ``(q, k, v, scale, rows)``),
    concatenation of the heads, output projection."""
    qkv = linear(x, w_qkv)
    q, k, v = split_qkv(qkv, H, d)
    q = rope(q, angles)
    k = rope(k, angles)
    S = q.shape[0]
    rows = np.arange(S) if rows is None else np.asarray(rows, dtype=np.int64)
    o = np.stack([attention_head(q[:, h], k[:, h], np.asarray(v[:, h], dtype=np.float64),
                                 scale, rows) for h in range(H)], axis=1)
    return linear(o.reshape(rows.size, H * d), w_o)
