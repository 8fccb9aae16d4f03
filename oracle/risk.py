"""Transition Risk Controller (Sec. 4.3, Eq. (6)-(10)), float64.

Readings of the terms the paper defines only in words (Sec. 4.3 names them
and defers their normalisations to the supplementary material):

* d_z     = sum|z_t - z_a| / (sum|z_a| + eps)   distance from the latest anchor
            (mean absolute values, as in Eq. (7); the element count cancels)
* d_age   = (n_s + 1) / (A_max + 1)             consecutive surrogate steps
* d_phase = |q_t - q_a|                         scheduler-phase displacement
* d_cam   = ||c_t - c_a|| / (||c_a|| + eps)     camera/motion change (0 if absent)
* d_depth = likewise for depth/geometry (0 if absent)
* u_phase = q_t (remaining-rollout fraction), u_cam = min(1, d_cam),
  u_depth = min(1, d_depth)
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def f64(a):
    return np.asarray(a, dtype=np.float64)


@dataclass
class Proxy:
    d_z: float
    d_age: float
    d_phase: float
    d_cam: float
    d_depth: float
    p: float


def local_proxy(z, z_anchor, n_s: int, q: float, q_a: float, p, d_cam: float = 0.0,
                d_depth: float = 0.0) -> Proxy:
    """p_t of Eq. (6). Without an anchor the anchor-relative terms are 0."""
    if z_anchor is None:
        dz, dph = 0.0, 0.0
    else:
        za = f64(z_anchor)
        dz = float(np.sum(np.abs(f64(z) - za)) / (np.sum(np.abs(za)) + p.eps))
        dph = abs(q - q_a)
    dage = (n_s + 1) / (p.age_max + 1)
    val = p.w_z * dz + p.w_age * dage + p.w_phase * dph + p.w_cam * d_cam + p.w_depth * d_depth
    return Proxy(dz, dage, dph, d_cam, d_depth, val)


def sensitivity_weight(q: float, p, d_cam: float = 0.0, d_depth: float = 0.0) -> float:
    """w_t of Eq. (9), capped at 2; 1 when future-impact weighting is switched off."""
    if not p.impact_weight:
        return 1.0
    u_cam, u_depth, u_phase = min(1.0, d_cam), min(1.0, d_depth), q
    return min(2.0, 1.0 + p.a_cam * u_cam + p.a_depth * u_depth + p.a_phase * u_phase)


def accumulate(R: float, eta: float, proxy: float, w: float, p):
    """Eq. (6), (9): d_hat = eta * p, Delta = w * d_hat, R_cand = lambda * R + Delta."""
    d_hat = eta * proxy
    delta = w * d_hat
    return d_hat, delta, p.lam * R + delta


def counterfactual_defect(z_exact, z_cf, eps: float) -> float:
    """Eq. (7): mean|z_exact - z_cf| / (mean|z_exact| + eps)."""
    ze = f64(z_exact)
    return float(np.mean(np.abs(ze - f64(z_cf))) / (np.mean(np.abs(ze)) + eps))


def calibrate(eta: float, d_cf: float, proxy: float, p) -> float:
    """Eq. (8): eta <- clamp(beta*eta + (1-beta)*d_cf/(p+eps), eta_min, eta_max)."""
    return float(np.clip(p.beta_d * eta + (1.0 - p.beta_d) * d_cf / (proxy + p.eps), p.eta_min, p.eta_max))


def available(bank_size: int, n_s: int, support: int, finite: bool, k: int, steps: int, p) -> bool:
    """Available_t (Sec. 4.3, reliability decision): non-empty memory, anchor age
    (consecutive surrogate commits) at most A_max, adequate support (unless the
    support constraint is switched off), finite candidate, and the step outside
    the mandatory-exact initial and final phases."""
    supported = support >= p.n_min or not p.support_constraint
    return (bank_size > 0 and n_s <= p.age_max and supported and finite
            and k >= p.k_init and k <= steps - 1 - p.k_ref)


def decide(avail: bool, r_cand: float, tau: float) -> bool:
    """Eq. (10): True = Surrogate iff Available and R_cand <= tau (inclusive)."""
    return bool(avail and r_cand <= tau)
