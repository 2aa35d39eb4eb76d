"""Property-based tests (hypothesis) of the layout maps, the chunk rule and
the time model, on the CPU.

The pack formula of Sec. 3.3 sends element (p, s, h0 + j, t) of the
sequence-sharded ``[P][S/P][H][d]`` tensor to (j, p S/P + s, t) of the chunk
``[H_c][S][d]``.  Here it is checked element by element with plain loops over
random small shapes, head ranges and element sizes, for the oracle's C
implementation; unpack is checked as its inverse on the chunk's heads and as
the identity elsewhere, and packs of adjacent head ranges compose.  The chunk
rule is checked for the properties Sec. 3.3 states (C parts, sizes differing by
at most one, larger first, summing to H) on the oracle and on the library's host
code.  The time model's best integer chunk count is checked against the real
optimum of the appendix's theorem.
"""
import math

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from oracle import time_model as tm

SETTINGS = settings(max_examples=150, deadline=None,
                    suppress_health_check=[HealthCheck.too_slow])
DTYPES = [np.uint8, np.uint16, np.float32, np.float64]


@st.composite
def layouts(draw):
    P = draw(st.integers(1, 5))
    S = P * draw(st.integers(1, 6))
    H = draw(st.integers(1, 6))
    d = draw(st.integers(1, 5))
    h0 = draw(st.integers(0, H - 1))
    Hc = draw(st.integers(1, H - h0))
    dt = draw(st.sampled_from(DTYPES))
    seed = draw(st.integers(0, 2**31 - 1))
    return P, S, H, d, h0, Hc, np.dtype(dt), seed


def random_tensor(shape, dt, seed):
    rng = np.random.default_rng(seed)
    if dt.kind == "u":
        return rng.integers(0, np.iinfo(dt).max, size=shape, endpoint=True).astype(dt)
    return rng.standard_normal(shape).astype(dt)


@SETTINGS
@given(layouts())
def test_pack_moves_every_element_by_the_formula(case):
    P, S, H, d, h0, Hc, dt, seed = case
    src = random_tensor((S, H, d), dt, seed)
    out = oracle.pack(src, P, h0, Hc)
    assert out.shape == (Hc, S, d) and out.dtype == dt
    shard = S // P
    sharded = src.reshape(P, shard, H, d)
    for j in range(Hc):
        for p in range(P):
            for s in range(shard):
                for t in range(d):
                    assert out[j, p * shard + s, t].tobytes() == sharded[p, s, h0 + j, t].tobytes()


@SETTINGS
@given(layouts())
def test_unpack_inverts_pack_and_leaves_other_heads(case):
    P, S, H, d, h0, Hc, dt, seed = case
    src = random_tensor((S, H, d), dt, seed)
    background = random_tensor((S, H, d), dt, seed + 1)
    back = oracle.unpack(oracle.pack(src, P, h0, Hc), background, P, h0)
    inside = np.zeros(H, dtype=bool)
    inside[h0:h0 + Hc] = True
    assert back[:, inside].tobytes() == src[:, inside].tobytes()
    assert back[:, ~inside].tobytes() == background[:, ~inside].tobytes()


@SETTINGS
@given(layouts(), st.data())
def test_packs_of_adjacent_head_ranges_compose(case, data):
    P, S, H, d, h0, Hc, dt, seed = case
    if Hc < 2:
        return
    split = data.draw(st.integers(1, Hc - 1))
    src = random_tensor((S, H, d), dt, seed)
    whole = oracle.pack(src, P, h0, Hc)
    parts = np.concatenate([oracle.pack(src, P, h0, split),
                            oracle.pack(src, P, h0 + split, Hc - split)])
    assert whole.tobytes() == parts.tobytes()


@SETTINGS
@given(st.integers(1, 5), st.integers(1, 6), st.integers(1, 4), st.integers(1, 3),
       st.integers(0, 2**31 - 1))
def test_pack_rejects_shapes_outside_the_formula(P, S, H, d, seed):
    src = random_tensor((P * S + 1, H, d), np.dtype(np.float32), seed)
    if P > 1:   # S not divisible by P
        with pytest.raises(ValueError):
            oracle.pack(src, P, 0, H)
    src = random_tensor((P * S, H, d), np.dtype(np.float32), seed)
    with pytest.raises(ValueError):
        oracle.pack(src, P, H - 1, 2)     # head range past H


@SETTINGS
@given(st.integers(1, 4096), st.data())
def test_chunk_rule_properties_and_library_agreement(H, data):
    import paper_2607_01817_amd as hcms
    C = data.draw(st.integers(1, min(H, 512)))
    sizes = oracle.default_chunks(H, C)
    assert len(sizes) == C and sum(sizes) == H
    assert max(sizes) - min(sizes) <= 1
    assert sizes == sorted(sizes, reverse=True)
    assert sizes.count(H // C + 1) == H % C
    offs = oracle.chunk_offsets(sizes)
    assert offs[0] == 0 and all(offs[c + 1] == offs[c] + sizes[c] for c in range(C - 1))
    assert hcms.default_chunks(H, C) == sizes


@SETTINGS
@given(st.floats(1e-3, 1e3), st.floats(1e-4, 1e2), st.integers(1, 64))
def test_best_integer_chunk_count_brackets_the_real_optimum(t_comm, beta, H):
    c_real, best = tm.optimal_chunks(t_comm, beta, H)
    assert c_real == pytest.approx(math.sqrt(t_comm / beta))
    cost = [t_comm / c + c * beta for c in range(1, H + 1)]
    # Brute force over every C in [1, H], ties to the smaller C.
    assert best == 1 + int(np.argmin(cost))
    # T is convex in C, so the best integer is the floor or ceiling of the
    # real optimum clamped into [1, H].
    lo = min(max(math.floor(c_real), 1), H)
    hi = min(max(math.ceil(c_real), 1), H)
    assert best in (lo, hi)
    # More chunks never help once C passes the real optimum.
    for c in range(max(best, math.ceil(c_real)), H):
        assert cost[c] >= cost[c - 1] - 1e-12 * max(cost)
