"""Oracle of the HCMS time model (arXiv 2607.01817, Sec. 3.7 and the appendix).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: the test suite and
``bench.py`` may call it; the product path never does.  Plain Python floats,
one function per equation of the paper, written from its definitions:

* :func:`hcms_time`      the appendix's HCMS time equation,
  T(C) = T_0 + T_comm / C + T_attn + C * beta;
* :func:`baseline_time`  the appendix's baseline, T_0 + T_comm + T_attn;
* :func:`optimal_chunks` the optimal-chunk theorem, C* = sqrt(T_comm / beta),
  and the best integer chunk count in [1, H] by evaluating T at every C;
* :func:`speedup`        the appendix's speedup equation,
  S(C) = 1 / (1 - rho (C - 1) / C + C beta / T_total);
* :func:`fit`            least squares of T(C) = a + b / C + beta C over
  measured points, by numpy's lstsq (the library routine is the step; the
  model is the paper's).

Pins in ``tests/test_time_model.py``: C* zeroes dT/dC and every integer
neighbour is no better; S(C) = T_base / T(C) with rho = T_comm / T_base;
S -> 1 / (1 - rho) as beta -> 0 and C grows (the paper's upper bound); S(1) =
1 / (1 + beta / T_total); fits recover planted parameters exactly.
"""
from __future__ import annotations

import math

import numpy as np


def hcms_time(t0: float, t_comm: float, t_attn: float, beta: float, C: int) -> float:
    return t0 + t_comm / C + t_attn + C * beta


def baseline_time(t0: float, t_comm: float, t_attn: float) -> float:
    return t0 + t_comm + t_attn


def optimal_chunks(t_comm: float, beta: float, H: int) -> tuple[float, int]:
    """(C*, the integer C in [1, H] with the smallest model time; ties go to
    the smaller C)."""
    c_real = math.sqrt(t_comm / beta) if beta > 0 else math.inf
    best = min(range(1, H + 1), key=lambda c: (t_comm / c + c * beta, c))
    return c_real, best


def speedup(rho: float, beta_over_total: float, C: int) -> float:
    return 1.0 / (1.0 - rho * (C - 1) / C + C * beta_over_total)


def fit(chunk_counts, times) -> tuple[float, float, float]:
    """(a, T_comm, beta) of the least-squares fit T(C) = a + T_comm / C + beta C."""
    c = np.asarray(chunk_counts, dtype=np.float64)
    A = np.stack([np.ones_like(c), 1.0 / c, c], axis=1)
    x, *_ = np.linalg.lstsq(A, np.asarray(times, dtype=np.float64), rcond=None)
    return float(x[0]), float(x[1]), float(x[2])
