"""Inference loop (Sec. 4.4): exact anchors plus risk-controlled surrogate steps.

The paper's complete algorithm sits in its missing supplementary material;
this loop assembles the steps Sec. 4.2-4.4 describe, in this order, for
k = 0..S-1 (the paper's t -> t-1 is k -> k+1, q_k = t_k):

1. Lift the current state with the pre-insertion history (Eq. (2)) and, if the
   bank holds a record, build the candidate z_hat (Eq. (3)-(5)).
2. Local proxy, sensitivity weight and candidate risk (Eq. (6), (9)).
3. Decision (Eq. (10)).
4. Surrogate: commit z_hat, R <- R_cand, one more consecutive surrogate step;
   never inserted into the bank.
   Exact: z_{k+1} = Psi(z_k, F_theta(z_k, t_k)); if the pre-insertion
   candidate was supported and finite, the counterfactual defect (Eq. (7))
   calibrates eta_d (Eq. (8)); R <- lambda*R; insert the record
   (phi_in = Phi(z_k; H_pre), phi_out = Phi(z_{k+1}; H_pre), both under the
   pre-insertion anchor and history), then the anchor becomes z_k with
   (q_a, q_{a-1}) = (t_k, t_{k+1}), h becomes the summary of this transition
   and the surrogate count resets.

Modes: "risk" (Eq. (10) as written), "forced" (decisions from a mask, with
unsupported candidates still falling back to exact), "periodic" (exact when
k mod period == 0, else the surrogate when available: the periodic placement
of the ablation study, Sec. 5.4), "all_exact", and the same loop with F_theta
replaced by recorded velocities (``replay_denoiser``). The surrogate
construction and the ablation switches come from the parameters.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional

import numpy as np

from . import risk as rk
from . import surrogate as sg
from .scheduler import psi, t_at


@dataclass
class StepLog:
    k: int
    t: float
    exact: bool
    bank: int
    support: int
    alpha: float
    pi: List[float]
    kappa: List[float]
    sims_in: List[float]
    finite: bool
    d_z: float
    d_age: float
    d_phase: float
    p: float
    d_hat: float
    w: float
    r_cand: float
    margin: float
    sim_margin: float
    available: bool
    d_cf: float
    eta: float          # eta_d after this step
    R: float            # R after this step
    slot: int           # bank slot written (-1 on surrogate steps)


@dataclass
class Result:
    z: np.ndarray
    schedule: List[int]               # 0 = exact, 1 = surrogate
    log: List[StepLog]
    calls: int                        # denoiser evaluations
    inserts: int


def rollout(denoise: Callable[[np.ndarray, int, float], np.ndarray], z_T, steps: int, p,
            mode: str = "risk", forced: Optional[List[int]] = None, cam=None,
            trace: Optional[list] = None) -> Result:
    """Run S denoising steps from z_T. ``denoise(z, k, t)`` returns v_k.
    ``forced[k]`` = 1 requests a surrogate step (mode "forced").
    ``trace``, if given, receives z_{k+1} after every step."""
    tau = {"risk": p.tau_risk, "all_exact": -np.inf}.get(mode, p.tau_risk)
    cam_desc = sg.cam_descriptor(cam, p.eps_nu)
    bank = sg.Bank(p.bank_capacity)
    z = np.asarray(z_T, dtype=np.float64)
    z_a, q_a, q_am1, h = None, 0.0, 0.0, None
    R, eta, n_s = p.r0, p.eta0, 0
    sched, logs, calls = [], [], 0
    for k in range(steps):
        t, tn = t_at(k, steps), t_at(k + 1, steps)
        phi = sg.lift(z, z_a, h, t, cam_desc, p)
        bank_before = len(bank)
        if p.surrogate == "secant":
            cand = sg.secant_candidate(z, z_a, bank, t, tn, q_a, q_am1, p)
        else:
            cand = sg.candidate(phi, bank, tn, q_a, q_am1, p, z=z)
        support = len(cand.support) if cand else 0
        finite = cand.finite if cand else False
        prox = rk.local_proxy(z, z_a, n_s, t, q_a, p)
        w = rk.sensitivity_weight(t, p)
        d_hat, _, r_cand = rk.accumulate(R, eta, prox.p, w, p)
        avail = rk.available(len(bank), n_s, support, finite, k, steps, p)
        if mode == "forced":
            take = bool(forced[k]) and avail
        elif mode == "periodic":
            take = k % p.period != 0 and avail
        else:
            take = rk.decide(avail, r_cand, tau)
        margin = abs(r_cand - tau) / max(abs(tau), 1e-12) if np.isfinite(tau) else np.inf
        sim_margin = (float(np.min(np.abs(cand.sims_in - p.theta_sim))) if cand else np.inf)
        d_cf, slot = float("nan"), -1
        if take:
            z_next = cand.z_hat
            R = r_cand
            n_s += 1
        else:
            v = np.asarray(denoise(z, k, t), dtype=np.float64)
            calls += 1
            z_next = psi(z, v, t, tn)
            supported = support >= p.n_min or not p.support_constraint
            if cand is not None and supported and finite:
                d_cf = rk.counterfactual_defect(z_next, cand.z_hat, p.eps)
                if p.calibrate:
                    eta = rk.calibrate(eta, d_cf, prox.p, p)
            R = p.lam * R
            phi_out = sg.lift(z_next, z_a, h, tn, cam_desc, p)
            slot = bank.insert(sg.Record(phi, phi_out, sg.summary(phi), sg.summary(phi_out), t, tn,
                                         z_next.copy()))
            h = sg.history_summary(z, z_next, p)
            z_a, q_a, q_am1 = z, t, tn
            n_s = 0
        sched.append(1 if take else 0)
        logs.append(StepLog(k, t, not take, bank_before, support, cand.alpha if cand else 0.0,
                            list(cand.pi) if cand else [], list(cand.kappa) if cand else [],
                            list(cand.sims_in) if cand else [], finite,
                            prox.d_z, prox.d_age, prox.d_phase, prox.p, d_hat, w, r_cand, margin,
                            sim_margin, avail, d_cf, eta, R, slot))
        z = z_next
        if trace is not None:
            trace.append(z.copy())
    return Result(z, sched, logs, calls, bank.inserts)


def dit_denoiser(W, cfg, inputs):
    """F_theta of the synthetic DiT as a rollout callback."""
    from .dit import dit_forward

    def f(z, k, t):
        return dit_forward(W, cfg, z, t, inputs.get("cond"), inputs.get("text"), inputs.get("cam"))
    return f


def replay_denoiser(vel):
    """Recorded velocities v_k in place of F_theta (control-path checks at large shapes)."""
    def f(z, k, t):
        return np.asarray(vel[k], dtype=np.float64)
    return f
