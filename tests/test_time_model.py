"""The HCMS time model: the oracle pinned by the paper and by closed forms, and
the C library checked against the oracle (CPU only)."""
import ctypes
import math
import random

import numpy as np
import pytest

import paper_2607_01817_amd as hcms
from oracle import time_model as tm

EARG, ECHUNKS, ESHAPE, ENULL = -7, -3, -2, -1


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
