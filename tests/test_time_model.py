"""The HCMS time model: the oracle pinned by the paper and by closed forms, and
the C library checked against the oracle (CPU only)."""
import ctypes
import json
import math
import os
import random

import numpy as np
import pytest

import paper_2607_01817_amd as hcms
from oracle import time_model as tm

EARG, ECHUNKS, ESHAPE, ENULL, EDTYPE = -7, -3, -2, -1, -4
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# Oracle pins
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("rho,printed", [(0.35, 1.54), (0.20, 1.25), (0.10, 1.11)])
def test_upper_bound_matches_printed_applicability_table(rho, printed):
    """The applicability table prints S_max at the band edges of rho; the
    speedup equation with beta -> 0 and C -> inf must give the same."""
    s = tm.speedup(rho, 0.0, 10**9)
    assert round(s, 2) == printed
    assert s == pytest.approx(1.0 / (1.0 - rho), rel=1e-8)


def test_optimal_chunks_zeroes_the_derivative():
    rng = random.Random(3)
    for _ in range(200):
        t_comm, beta = rng.uniform(0.1, 50.0), rng.uniform(0.01, 5.0)
        c_star, _ = tm.optimal_chunks(t_comm, beta, 100)
        assert c_star == pytest.approx(math.sqrt(t_comm / beta))
        f = lambda c: tm.hcms_time(1.0, t_comm, 2.0, beta, c)  # noqa: E731
        h = 1e-5 * c_star
        assert (f(c_star + h) - f(c_star - h)) / (2 * h) == pytest.approx(0.0, abs=1e-6)
        assert f(c_star) <= min(f(c_star * 0.9), f(c_star * 1.1))


def test_best_integer_is_next_to_the_real_optimum():
    rng = random.Random(4)
    for _ in range(500):
        t_comm, beta, H = rng.uniform(0.0, 40.0), rng.uniform(0.001, 3.0), rng.randint(1, 48)
        c_star, best = tm.optimal_chunks(t_comm, beta, H)
        lo = min(max(math.floor(c_star), 1), H)
        assert best in (lo, min(lo + 1, H))


def test_speedup_is_baseline_over_hcms_time():
    """Two equations of the appendix must agree: S(C) = T_base / T_hcms(C)
    with rho = T_comm / T_base and beta / T_total = beta / T_base."""
    rng = random.Random(5)
    for _ in range(200):
        t0, t_comm, t_attn = rng.uniform(0, 5), rng.uniform(0, 20), rng.uniform(1, 50)
        beta, C = rng.uniform(0, 1), rng.randint(1, 40)
        base = tm.baseline_time(t0, t_comm, t_attn)
        s = tm.speedup(t_comm / base, beta / base, C)
        assert s == pytest.approx(base / tm.hcms_time(t0, t_comm, t_attn, beta, C), rel=1e-12)


def test_theory_validation_row_predicts_five_chunks():
    """Row 1 of the appendix's theory-validation table: rho = 39.6 %,
    beta = 1.41 ms on the 8-GPU RTX 5090 56K configuration, whose baseline
    time is 73.3 ms (sequence-scaling table).  T_comm = rho T_total gives
    C* = sqrt(T_comm / beta) = 4.54, and the best integer count is 5, the
    table's predicted (and measured) optimum."""
    g = json.load(open(os.path.join(GOLDEN, "theory_validation.json")))
    t_comm = g["rho"] * g["t_total_ms"]
    c_real, best = tm.optimal_chunks(t_comm, g["beta_ms"], g["H"])
    assert c_real == pytest.approx(4.5376, abs=1e-3)
    assert best == g["c_star_predicted"] == g["c_star_measured"]
    assert hcms.model_optimal_chunks(t_comm, g["beta_ms"], g["H"]) == (5, pytest.approx(c_real))
    # 4 and 6 chunks are worse than 5 in the model (the integer neighbours).
    f = lambda c: tm.hcms_time(0.0, t_comm, 0.0, g["beta_ms"], c)  # noqa: E731
    assert f(5) < f(4) < f(6)


def test_one_chunk_pays_only_its_overhead():
    for b in (0.0, 0.01, 0.3):
        assert tm.speedup(0.4, b, 1) == pytest.approx(1.0 / (1.0 + b))


def test_fit_recovers_planted_parameters():
    cs = [1, 2, 3, 4, 5, 8]
    for a, t_comm, beta in ((7.0, 0.1, 0.006), (40.0, 12.0, 1.4), (0.0, 0.0, 0.0)):
        ts = [a + t_comm / c + beta * c for c in cs]
        got = tm.fit(cs, ts)
        assert got == pytest.approx((a, t_comm, beta), abs=1e-9)


# ---------------------------------------------------------------------------
# Library against the oracle
# ---------------------------------------------------------------------------
def test_library_matches_oracle():
    rng = random.Random(6)
    for _ in range(300):
        t0, t_comm, t_attn = rng.uniform(0, 5), rng.uniform(0, 20), rng.uniform(0, 50)
        beta, C, H = rng.uniform(0, 2), rng.randint(1, 64), rng.randint(1, 64)
        assert hcms.model_time(t0, t_comm, t_attn, beta, C) == \
            pytest.approx(tm.hcms_time(t0, t_comm, t_attn, beta, C), rel=1e-14)
        best, c_real = hcms.model_optimal_chunks(t_comm, beta, H)
        o_real, o_best = tm.optimal_chunks(t_comm, beta, H)
        assert best == o_best
        assert c_real == pytest.approx(o_real, rel=1e-14)
        rho, b = rng.uniform(0, 1), rng.uniform(0, 0.1)
        assert hcms.model_speedup(rho, b, C) == pytest.approx(tm.speedup(rho, b, C), rel=1e-14)


def test_library_fit_matches_oracle_on_noisy_points():
    rng = np.random.default_rng(7)
    for n in (3, 5, 10, 40):
        cs = list(range(1, n + 1))
        ts = [3.0 + 2.0 / c + 0.05 * c + rng.normal(0, 0.01) for c in cs]
        assert hcms.model_fit(cs, ts) == pytest.approx(tm.fit(cs, ts), rel=1e-9, abs=1e-9)


def test_zero_overhead_picks_every_head():
    assert hcms.model_optimal_chunks(5.0, 0.0, 12) == (12, math.inf)
    assert tm.optimal_chunks(5.0, 0.0, 12) == (math.inf, 12)


def test_library_validation():
    lib = hcms.load()
    out = ctypes.c_double()
    assert lib.hcms_model_time(0, 1, 1, 0.1, 0, ctypes.byref(out)) == ECHUNKS
    assert lib.hcms_model_time(0, -1, 1, 0.1, 2, ctypes.byref(out)) == EARG
    assert lib.hcms_model_time(0, float("nan"), 1, 0.1, 2, ctypes.byref(out)) == EARG
    assert lib.hcms_model_time(0, 1, 1, 0.1, 2, None) == ENULL
    assert lib.hcms_model_optimal_chunks(1.0, 0.1, 0, None) == ESHAPE
    assert lib.hcms_model_optimal_chunks(1.0, -0.1, 4, None) == EARG
    assert lib.hcms_model_speedup(1.5, 0.0, 2, ctypes.byref(out)) == EARG
    assert lib.hcms_model_speedup(0.5, 0.0, 0, ctypes.byref(out)) == ECHUNKS
    cs = (ctypes.c_int * 3)(1, 1, 1)
    ts = (ctypes.c_double * 3)(1.0, 1.0, 1.0)
    a, b, c = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    assert lib.hcms_model_fit(cs, ts, 3, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)) == EARG
    assert lib.hcms_model_fit(cs, ts, 2, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)) == EARG
    cs0 = (ctypes.c_int * 3)(0, 1, 2)
    assert lib.hcms_model_fit(cs0, ts, 3, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)) == ECHUNKS


# ---------------------------------------------------------------------------
# One GPU: attention time through the rounds of each launch
# ---------------------------------------------------------------------------
def test_round_identity():
    """With g0 = 1 a launch costs its round count ceil(W / n); the sum over
    launches splits as sum W / n plus the idle share of the partial rounds."""
    rng = random.Random(8)
    for _ in range(500):
        n = rng.randint(1, 300)
        Ws = [rng.randint(1, 3000) for _ in range(rng.randint(1, 8))]
        R = sum(-(-w // n) for w in Ws)
        assert sum(tm.launch_rounds(w, n, 1.0) for w in Ws) == pytest.approx(R)
        idle = sum((n - w % n) % n for w in Ws) / n
        assert R == pytest.approx(sum(Ws) / n + idle)
        g0 = rng.uniform(0.05, 1.0)
        # The partial rounds cost g0 of their idle share: T = sum W / n + g0 idle.
        assert sum(tm.launch_rounds(w, n, g0) for w in Ws) == pytest.approx(sum(Ws) / n + g0 * idle)


def test_one_gpu_model_reduces_to_the_paper_model():
    """Launches that fill whole rounds keep the attention time fixed; the
    pipelined plan of C equal chunks is then the appendix's T_hcms(C) with
    T_comm = 4 H t_copy (pack 3 tensors, unpack 1), per-chunk overhead
    beta' = 2 beta + drain t_round and T_0 = 3 beta."""
    n, br = 256, 256
    for H, S in ((8, 256 * 64), (12, 256 * 128)):
        tiles = S // br
        for C in (c for c in range(1, H + 1) if H % c == 0 and (tiles * (H // c)) % n == 0):
            sizes = [H // C] * C
            t_round, t_copy, beta = 0.9, 0.004, 0.006
            drain = 0.02
            got = tm.plan_time(S, sizes, tm.PIPELINED if C > 1 else tm.SERIAL, n, br, t_round,
                               0.5, t_copy, beta, True, drain)
            t_attn = t_round * tiles * H / n
            if C == 1:
                assert got == pytest.approx(t_attn + 4 * H * t_copy + drain * t_round)
            else:
                assert got == pytest.approx(tm.hcms_time(3 * beta, 4 * H * t_copy, t_attn,
                                                         2 * beta + drain * t_round, C))


def test_worked_rounds_of_the_wan_p4_share():
    """Wan-P4 (S = 32760, 10 heads, 256-query tiles: 128 per head) on 256
    slots, chunks 5 + 5: each launch is 640 workgroups = 2 full rounds and a
    half-full one; two lanes pool them into 1280 = 5 full rounds.  One lane:
    2 (2 + g0 + (1 - g0) / 2) rounds.  Copies: serial moves all 40
    head-tensors on the path, the other plans chunk 0's pack (15) and the
    last unpack (5); the fused plan also the copies of launches that leave
    fewer than 32 slots idle (none here: 128 idle)."""
    g0, tr, tc, b = 0.4, 1.0, 0.01, 0.1
    one_lane = 2 * (2 + g0 + (1 - g0) / 2)
    S, sizes = 32760, (5, 5)
    assert tm.plan_time(S, sizes, tm.SERIAL, 256, 256, tr, g0, tc, b) == pytest.approx(one_lane + 0.4)
    assert tm.plan_time(S, sizes, tm.LANES, 256, 256, tr, g0, tc, b) == pytest.approx(5 + 0.2 + 0.4)
    assert tm.plan_time(S, sizes, tm.FUSED, 256, 256, tr, g0, tc, b) == pytest.approx(one_lane + 0.2)
    assert tm.plan_time(S, sizes, tm.INLINE, 256, 256, tr, g0, tc, b) == pytest.approx(one_lane + 0.6)
    assert tm.plan_time(S, sizes, tm.PIPELINED, 256, 256, tr, g0, tc, b) == pytest.approx(
        one_lane + 0.2 + 0.7)
    # Chunks 2 x 5 fill one round each and leave no slot idle: the fused plan
    # carries nothing, so every copy is on the path, as in the serial plan.
    fused = tm.plan_time(S, (2,) * 5, tm.FUSED, 256, 256, tr, g0, tc, b)
    assert fused == pytest.approx(5 + 40 * tc)
    assert fused == pytest.approx(tm.plan_time(S, (2,) * 5, tm.SERIAL, 256, 256, tr, g0, tc, b))


def test_worked_split_tails():
    """The kernel splits a launch's last round by key segments.  Wan-P8 in
    one chunk (S = 56160: 220 tiles per head, 878 key blocks): 1100
    workgroups = 4 full rounds and 76 tiles; 3 x 76 = 228 <= 256, so three
    ways, a round a third as long with 228 of 256 slots busy.  Wan-P4 in
    5 + 5 (S = 32760): 640 = 2 rounds and 128 tiles, 2 x 128 = 256: two ways,
    two thirds of a full round.  Wan-P8 in 2 + 2 + 1: 440 = 256 + 184 and
    220, no split fits.  Keys of fewer than 12 blocks are never split."""
    g0 = 0.4
    assert tm.tail_ways(1100, 256, 56160, True) == 3
    assert tm.launch_rounds(1100, 256, g0, 3) == pytest.approx(4 + (g0 + (1 - g0) * 228 / 256) / 3)
    assert tm.plan_time(56160, (5,), tm.SERIAL, 256, 256, 1.0, g0, 0.0, 0.0, True) == \
        pytest.approx(4 + (g0 + (1 - g0) * 228 / 256) / 3)
    assert tm.tail_ways(640, 256, 32760, True) == 2
    assert tm.plan_time(32760, (5, 5), tm.SERIAL, 256, 256, 1.0, g0, 0.0, 0.0, True) == \
        pytest.approx(2 * (2 + 2 / 3))
    assert tm.tail_ways(440, 256, 56160, True) == 1 and tm.tail_ways(220, 256, 56160, True) == 1
    assert tm.tail_ways(1100, 256, 56160, False) == 1
    assert tm.tail_ways(1100, 256, 64 * 11, True) == 1
    # Lanes pool 2 + 2 + 1 into the one-chunk launch's 1100 workgroups; the
    # lanes' last launches split the 76 tiles past the 4 pooled rounds, so
    # the attention takes what the one-chunk launch takes (two drains).
    assert tm.plan_time(56160, (2, 2, 1), tm.LANES, 256, 256, 1.0, g0, 0.0, 0.0, True) == \
        pytest.approx(4 + (g0 + (1 - g0) * 228 / 256) / 3)
    assert tm.plan_time(56160, (2, 2, 1), tm.LANES, 256, 256, 1.0, g0, 0.0, 0.0, False) == \
        pytest.approx(4 + g0 + (1 - g0) * 76 / 256)


def _plan_of(S, d, dtype=0, n_cu=256):
    return lambda sizes: hcms.auto_mode(S, d, sizes, n_cu, dtype=dtype)


@pytest.mark.parametrize("S,H,d", [(56160, 5, 128), (32760, 10, 128), (100000, 40, 128),
                                   (4096, 8, 128), (8192, 16, 64), (1000, 3, 64)])
def test_plan_time_and_choice_match_oracle(S, H, d):
    rng = random.Random(S + H)
    br = 256 if d == 128 else 128
    n = 256 if d == 128 else 512
    for _ in range(20):
        t_round, g0 = rng.uniform(0.01, 2.0), rng.uniform(0.05, 1.0)
        t_copy, beta = rng.uniform(0.0, 0.02), rng.uniform(0.0, 0.02)
        for C in range(1, H + 1):
            sizes = hcms.default_chunks(H, C)
            for mode in (hcms.MODE_SERIAL, hcms.MODE_PIPELINED, hcms.MODE_INLINE, hcms.MODE_LANES,
                         hcms.MODE_SLOTS, hcms.MODE_FUSED):
                got = hcms.model_plan_time(S, d, sizes, mode, 256, t_round, g0, t_copy, beta)
                want = tm.plan_time(S, sizes, mode, n, br, t_round, g0, t_copy, beta, d == 128)
                assert got == pytest.approx(want, rel=1e-12)
            auto = hcms.model_plan_time(S, d, sizes, hcms.MODE_AUTO, 256, t_round, g0, t_copy, beta)
            assert auto == pytest.approx(tm.plan_time(S, sizes, _plan_of(S, d)(sizes), n, br,
                                                      t_round, g0, t_copy, beta, d == 128),
                                         rel=1e-12)
        sizes, mode, t = hcms.choose_chunks(S, H, d, 256, t_round, g0, t_copy, beta)
        o_sizes, o_t = tm.choose_chunks(S, H, _plan_of(S, d), n, br, t_round, g0, t_copy, beta,
                                        split=d == 128)
        assert sizes == o_sizes and t == pytest.approx(o_t, rel=1e-12)
        assert mode == _plan_of(S, d)(sizes)
        # brute force over every C: nothing is faster than the choice
        for C in range(1, H + 1):
            s2 = hcms.default_chunks(H, C)
            assert hcms.model_plan_time(S, d, s2, hcms.MODE_AUTO, 256, t_round, g0, t_copy,
                                        beta) >= t - 1e-12


def test_choice_with_costly_synchronisation_is_one_chunk():
    """When a synchronisation costs more than the copies it could hide and
    every launch fills whole rounds, one chunk (serial) is fastest."""
    sizes, mode, _ = hcms.choose_chunks(32768, 8, 128, 256, 1.0, 0.5, 0.001, 1.0)
    assert sizes == [8] and mode == hcms.MODE_SERIAL


def test_one_gpu_model_validation():
    lib = hcms.load()
    out = ctypes.c_double()
    sz = (ctypes.c_int * 2)(2, 3)
    f = lib.hcms_model_plan_time
    o = ctypes.byref(out)
    assert f(100, 128, 0, sz, 2, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, None) == ENULL
    assert f(100, 96, 0, sz, 2, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, o) == ESHAPE
    assert f(100, 128, 3, sz, 2, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, o) == EDTYPE
    assert f(100, 128, 0, sz, 2, 9, 256, 1.0, 0.5, 0.0, 0.0, 0.0, o) == EARG
    assert f(100, 128, 0, sz, 2, 0, 256, 1.0, 0.0, 0.0, 0.0, 0.0, o) == EARG
    assert f(100, 128, 0, sz, 2, 0, 256, 1.0, 1.5, 0.0, 0.0, 0.0, o) == EARG
    assert f(100, 128, 0, sz, 2, 0, 256, 1.0, 0.5, -0.1, 0.0, 0.0, o) == EARG
    assert f(100, 128, 0, sz, 2, 0, 0, 1.0, 0.5, 0.0, 0.0, 0.0, o) == EARG
    assert f(100, 128, 0, sz, 2, 0, 256, -1.0, 0.5, 0.0, 0.0, 0.0, o) == EARG
    assert f(100, 128, 0, sz, 0, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, o) == ECHUNKS
    bad = (ctypes.c_int * 2)(2, 0)
    assert f(100, 128, 0, bad, 2, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, o) == ECHUNKS
    buf = (ctypes.c_int * 4)()
    c = lib.hcms_choose_chunks
    assert c(100, 0, 128, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, 4, buf, None, None) == ESHAPE
    assert c(100, 4, 128, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, 0, buf, None, None) == ECHUNKS
    assert c(100, 4, 128, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, 4, None, None, None) == ENULL
    assert c(100, 4, 128, 0, 256, 1.0, 0.5, 0.0, 0.0, 0.0, 2, buf, None, None) in (1, 2)


def test_drain_adds_per_launch():
    """Each attention launch on the critical path adds `drain` rounds: C of
    them in one lane, ceil(C / 2) in two alternating lanes."""
    S, sizes = 32760, (2,) * 5        # five launches of one whole round each
    for mode, launches in ((tm.SERIAL, 5), (tm.FUSED, 5), (tm.PIPELINED, 5), (tm.LANES, 3)):
        a = tm.plan_time(S, sizes, mode, 256, 256, 1.0, 0.5, 0.01, 0.002, True, 0.0)
        b = tm.plan_time(S, sizes, mode, 256, 256, 1.0, 0.5, 0.01, 0.002, True, 0.03)
        assert b - a == pytest.approx(0.03 * launches)


def test_drain_library_matches_oracle():
    S = 32760
    rng = random.Random(9)
    for _ in range(50):
        dr = rng.uniform(0, 0.05)
        for C in range(1, 11):
            sz = hcms.default_chunks(10, C)
            for mode in (hcms.MODE_SERIAL, hcms.MODE_LANES, hcms.MODE_FUSED, hcms.MODE_PIPELINED):
                got = hcms.model_plan_time(S, 128, sz, mode, 256, 0.8, 0.4, 0.003, 0.006, drain=dr)
                want = tm.plan_time(S, sz, mode, 256, 256, 0.8, 0.4, 0.003, 0.006, True, dr)
                assert got == pytest.approx(want, rel=1e-12)
        sizes2, _, t = hcms.choose_chunks(S, 10, 128, 256, 0.8, 0.4, 0.003, 0.006, drain=dr)
        o = tm.choose_chunks(S, 10, _plan_of(S, 128), 256, 256, 0.8, 0.4, 0.003, 0.006,
                             split=True, drain=dr)
        assert sizes2 == o[0] and t == pytest.approx(o[1], rel=1e-12)
