"""Synthetic risk diagnostics, float64 (test infrastructure only).

Injection experiment of Observation 1 (Sec. 3): start from the exact
trajectory, replace the transition at step t by the surrogate once, and resume
exact inference. Recorded per step t:

* d_t: the local defect of the injected transition, Eq. (7) applied to the
  candidate built at z_t against the exact z_{t+1};
* D_t^down: the downstream degradation of the final latent,
  mean|z'_0 - z_0| / (mean|z_0| + eps), against the all-exact rollout;
* d_hat_t and Delta_t = w_t * d_hat_t (Eq. (6), (9)) as the controller sees them.

Predicted-vs-counterfactual agreement at exact anchors (Sec. 4.3): the pairs
(d_hat_t, d_cf_t) of an all-exact rollout.

False-safe rate: a criterion deems a step safe when it is at most its median;
the step is false-safe when its D^down also exceeds the median D^down (rates
overall and per third of the phase range; the thresholds are a reading, the
paper's tau_d and tau_D are not given).
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np

from . import rollout as ro


def _mean_abs_rel(a, b, eps):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.mean(np.abs(a - b)) / (np.mean(np.abs(b)) + eps))


def injection_sweep(denoise, z_T, steps: int, p, cam=None) -> Dict[str, list]:
    ref = ro.rollout(denoise, z_T, steps, p, mode="all_exact", cam=cam)
    trace_ref = []
    ro.rollout(denoise, z_T, steps, p, mode="all_exact", cam=cam, trace=trace_ref)
    out = {k: [] for k in ("step", "phase", "d_local", "d_hat", "delta", "down", "anchor_d_hat", "anchor_d_cf")}
    for lg in ref.log:
        if np.isfinite(lg.d_cf):
            out["anchor_d_hat"].append(lg.d_hat)
            out["anchor_d_cf"].append(lg.d_cf)
    for t in range(1, steps):
        if not ref.log[t].available:
            continue
        mask = [0] * steps
        mask[t] = 1
        trace = []
        res = ro.rollout(denoise, z_T, steps, p, mode="forced", forced=mask, cam=cam, trace=trace)
        assert res.schedule == mask
        lg = res.log[t]
        out["step"].append(t)
        out["phase"].append(lg.t)
        # the injected transition z_t -> z_hat against the exact z_{t+1}
        out["d_local"].append(_mean_abs_rel(trace[t], trace_ref[t], p.eps))
        out["d_hat"].append(lg.d_hat)
        out["delta"].append(lg.w * lg.d_hat)
        out["down"].append(_mean_abs_rel(res.z, ref.z, p.eps))
    return out


def pearson(x, y) -> float:
    x, y = np.asarray(x, np.float64), np.asarray(y, np.float64)
    mx, my = x.mean(), y.mean()
    return float(np.sum((x - mx) * (y - my)) / np.sqrt(np.sum((x - mx) ** 2) * np.sum((y - my) ** 2)))


def average_ranks(x) -> np.ndarray:
    """Rank of each value (1 = smallest); equal values get the mean of their ranks."""
    x = np.asarray(x, np.float64)
    r = np.empty(len(x))
    for i, v in enumerate(x):
        less = np.sum(x < v)
        equal = np.sum(x == v)
        r[i] = less + (equal + 1) / 2.0
    return r


def spearman(x, y) -> float:
    return pearson(average_ranks(x), average_ranks(y))


def false_safe_rates(criterion, down, phase, bins: int = 3) -> Dict[str, float]:
    c, d, q = (np.asarray(a, np.float64) for a in (criterion, down, phase))
    c_med, d_med = np.median(c), np.median(d)
    rates = {}
    groups: List[tuple] = [("all", np.ones(len(c), bool))]
    for b in range(bins):
        lo, hi = b / bins, (b + 1) / bins
        sel = (q >= lo) & ((q < hi) if b < bins - 1 else (q <= hi))
        groups.append((f"phase_bin{b}", sel))
    for name, sel in groups:
        deemed_safe = [i for i in range(len(c)) if sel[i] and c[i] <= c_med]
        if not deemed_safe:
            rates[name] = float("nan")
            continue
        rates[name] = sum(1 for i in deemed_safe if d[i] > d_med) / len(deemed_safe)
    return rates
