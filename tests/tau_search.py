"""Risk thresholds for rollout parity cases, chosen from the oracle alone.

A rollout's schedule stays the same for every threshold tau in [a, b), with
a the largest R_cand of a step that took the surrogate and b the smallest
R_cand of an available step that stayed exact (Eq. (10): surrogate iff
available and R_cand <= tau): no decision changes inside that interval, so
neither does any later state. ``explore`` covers a range of thresholds with
such intervals, one oracle rollout per interval; ``pick`` takes, for a wanted
number of surrogate steps, the schedule whose interval is widest relative to
its centre and puts tau there, which makes the relative margin
min_k |R_cand_k - tau| / tau as large as the schedules allow. Test
infrastructure: it calls only the oracle.
"""
from __future__ import annotations

import hashlib
import math
from typing import Callable, Dict, List, Tuple

import numpy as np


def interval(res) -> Tuple[float, float]:
    """[a, b) of thresholds that reproduce ``res``'s schedule."""
    a = max((l.r_cand for l, s in zip(res.log, res.schedule) if s == 1), default=0.0)
    b = min((l.r_cand for l, s in zip(res.log, res.schedule) if s == 0 and l.available), default=math.inf)
    return a, b


def centre(a: float, b: float) -> float:
    if math.isinf(b):
        return 4.0 * a if a > 0 else 1.0
    return 0.5 * (a + b)


def margin(res, tau: float) -> float:
    """Smallest relative distance of an available step's R_cand from tau."""
    return min((abs(l.r_cand - tau) / tau for l in res.log if l.available), default=math.inf)


def memo_denoiser(den: Callable, cache: Dict) -> Callable:
    """The same denoiser with its evaluations cached by (k, latent bytes): rollouts
    at different thresholds share their exact prefix."""
    def f(z, k, t):
        key = (k, hashlib.blake2b(np.ascontiguousarray(z).tobytes(), digest_size=16).hexdigest())
        if key not in cache:
            cache[key] = np.asarray(den(z, k, t), dtype=np.float64)
        return cache[key]
    return f


def explore(run: Callable, lo: float = 1e-4, hi: float = 1e2, budget: int = 40, gap: float = 1.02,
            log=None, targets=(), min_margin: float = math.inf, known=()) -> List[Tuple[float, float, int, list]]:
    """Schedules over thresholds [lo, hi]: a list of (a, b, surrogate count,
    schedule). Probes the geometric centre of the widest threshold range no
    visited interval covers, until every uncovered range is narrower than the
    ratio ``gap``, ``budget`` rollouts have run, or every count in ``targets``
    has a schedule with a margin of at least ``min_margin``. ``known``:
    schedules of earlier rollouts (same tuple form), whose ranges are skipped."""
    seen: List[Tuple[float, float, int, list]] = list(known)
    todo = [(lo, hi)]
    for a, b, _, _ in known:                 # ranges earlier rollouts already cover
        nxt = []
        for x, y in todo:
            if b <= x or a >= y:
                nxt.append((x, y))
                continue
            if a > x:
                nxt.append((x, a))
            if b < y:
                nxt.append((b * (1 + 1e-12), y))
        todo = nxt
    for _ in range(budget):
        if not todo:
            break
        if targets and all(pick(seen, n)[1] >= min_margin for n in targets):
            break
        todo.sort(key=lambda r: r[1] / r[0])
        x, y = todo.pop()
        if y / x < gap:
            break
        tau = math.sqrt(x * y)
        res = run(tau)
        a, b = interval(res)
        n = sum(res.schedule)
        seen.append((a, b, n, list(res.schedule)))
        if log:
            log(f"tau {tau:.6g}: {n} surrogate steps, interval [{a:.6g}, {b:.6g})")
        # the part of [x, y) not covered by [a, b) is still unexplored
        if a > x:
            todo.append((x, a))
        if b < y:
            todo.append((b * (1 + 1e-12), y))
    return seen


def pick(seen, n_target: int) -> Tuple[float, float]:
    """(tau, relative margin) for the visited schedule with ``n_target`` surrogate
    steps whose interval gives the largest margin; (nan, 0) if there is none."""
    best = (math.nan, 0.0)
    for a, b, n, _ in seen:
        if n != n_target:
            continue
        tau = centre(a, b)
        m = min((tau - a) / tau if a > 0 else math.inf, (b - tau) / tau if math.isfinite(b) else math.inf)
        if m > best[1]:
            best = (tau, m)
    return best
