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

The one-GPU extension (this library's reading; the paper holds the attention
time fixed):

* :func:`launch_rounds`  duration, in full rounds, of a launch of W
  workgroups on n slots: floor(W / n) full rounds plus, when n does not
  divide W, one partial round with a fraction f of the slots busy lasting
  g0 + (1 - g0) f of a full one;
* :func:`tail_ways`      how many workgroups share each tile of a launch's
  last round when the kernel splits it by key segments;
* :func:`plan_time`      that attention time summed over the launches (the
  lanes plan pools the chunks' workgroups), plus the copies a plan leaves on
  the critical path times t_copy, plus its synchronisations times beta;
* :func:`choose_chunks`  the chunk count of the chunk rule whose plan the
  model predicts fastest, by evaluating every C.

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


# ---------------------------------------------------------------------------
# One GPU: the attention time depends on the chunking through its rounds
# ---------------------------------------------------------------------------
SERIAL, PIPELINED, INLINE, LANES, AUTO, SLOTS, FUSED = 0, 1, 2, 3, 4, 5, 6


def launch_rounds(W: int, n: int, g0: float, ways: int = 1) -> float:
    """Full rounds of a launch of W workgroups on n slots, the last one
    counted as g0 + (1 - g0) f of a round when only a fraction f of the slots
    has work.  With its last round's tiles split ``ways`` = 2 or 3 ways by key
    segments, that round holds ways times as many workgroups, each doing a
    share of the work: it lasts 2/3 (two ways: segments 0-1 and 2) or 1/3
    (three ways) as long."""
    full, rem = divmod(W, n)
    if rem == 0:
        return float(full)
    f = rem * ways / n
    length = {1: 1.0, 2: 2.0 / 3.0, 3: 1.0 / 3.0}[ways]
    return full + length * (g0 + (1.0 - g0) * f)


def tail_ways(W: int, n: int, S: int, split: bool) -> int:
    """How many workgroups share each tile of a launch's last round: 3 when
    three times its rem = W mod n tiles fit in one round, else 2 when twice
    do, else 1; only when ``split`` (a kernel that splits) and the keys span
    at least 12 blocks of 64 (three segments)."""
    rem = W % n
    if not split or rem == 0 or -(-S // 64) < 12:
        return 1
    return 3 if 3 * rem <= n else 2 if 2 * rem <= n else 1


def plan_time(S: int, sizes, mode: int, n_slots: int, queries_per_wg: int, t_round: float,
              g0: float, t_copy: float, beta: float, split: bool = False,
              drain: float = 0.0) -> float:
    """Model time of one plan of the chunk sizes ``sizes`` on one GPU with
    ``n_slots`` attention workgroups per round of ``queries_per_wg`` queries;
    ``split``: the attention kernel splits its launches' last rounds (the
    lanes plan splits the partial round of the pooled workgroups, in the
    lanes' last launches); ``drain``: rounds each attention
    launch on the critical path adds while its last workgroups finish (C of
    them in one lane, ceil(C / 2) when two lanes alternate)."""
    sizes = list(sizes)
    C, H = len(sizes), sum(sizes)
    tiles = -(-S // queries_per_wg)
    W = [tiles * h for h in sizes]
    if C == 1:
        mode = SERIAL
    if mode == LANES:
        attn = launch_rounds(sum(W), n_slots, g0, tail_ways(sum(W), n_slots, S, split))
        attn += drain * math.ceil(C / 2)
    else:
        attn = sum(launch_rounds(w, n_slots, g0, tail_ways(w, n_slots, S, split)) for w in W)
        attn += drain * C
    if mode == SERIAL:
        copies = 4 * H                    # 3 tensors packed, 1 unpacked, per head
    else:
        copies = 3 * sizes[0] + sizes[-1]
        if mode == FUSED:
            for c, w in enumerate(W):
                w_run = (w - w % n_slots) + (w % n_slots) * tail_ways(w, n_slots, S, split)
                idle = (n_slots - w_run % n_slots) % n_slots
                if idle >= max(1, n_slots // 8):
                    continue              # this launch carries its neighbours' copies
                if c + 1 < C:
                    copies += 3 * sizes[c + 1]
                if c >= 1:
                    copies += sizes[c - 1]
    syncs = {SERIAL: 0, FUSED: 0, INLINE: 4, LANES: 4, PIPELINED: 2 * C + 3, SLOTS: 2 * C + 3}[mode]
    return attn * t_round + copies * t_copy + syncs * beta


def choose_chunks(S: int, H: int, plan_of, n_slots: int, queries_per_wg: int, t_round: float,
                  g0: float, t_copy: float, beta: float, max_chunks: int | None = None,
                  split: bool = False, drain: float = 0.0):
    """(sizes, model time) of the fastest chunk count of the chunk rule, each
    C in the plan ``plan_of(sizes)`` picks; ties go to fewer chunks."""
    best = None
    for C in range(1, min(H, max_chunks or H) + 1):
        sizes = [H // C + (1 if c < H % C else 0) for c in range(C)]   # Sec. 3.3 chunk rule
        t = plan_time(S, sizes, plan_of(sizes), n_slots, queries_per_wg, t_round, g0, t_copy, beta,
                      split, drain)
        if best is None or t < best[1]:
            best = (sizes, t)
    return best
