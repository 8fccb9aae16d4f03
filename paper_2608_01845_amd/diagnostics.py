"""Synthetic risk diagnostics and the matched-budget controller/surrogate
factorization, run through the C ABI (every rollout step in the library's
kernels; only statistics over the returned logs and latents happen here).

Injection sweep (Observation 1, Sec. 3): from the exact trajectory, step t
takes the surrogate once and every other step is exact (a forced rollout with
a one-hot mask). Per injected step:

* d_t, the local defect of that transition: the counterfactual defect of
  Eq. (7) of step t's candidate on the all-exact trajectory (the state z_t is
  the same in both runs, so this is exactly the defect of the injected step);
* D_t^down, the downstream degradation: mean|z'_0 - z_0| / (mean|z_0| + eps)
  between the final latents of the injected and the all-exact rollouts;
* d_hat_t (Eq. (6), predicted defect) and Delta_t = w_t d_hat_t (Eq. (9)).

Agreement of the predicted defect with the counterfactual defect at exact
anchors (Sec. 4.3, calibration): Pearson/Spearman over every exact step whose
candidate was supported.

False-safe rate of a criterion (Observation 1): the criterion deems step t
safe when its value is at most its median over the sweep; a false-safe step is
deemed safe while its D^down exceeds the median D^down. Rates are reported
over all injected steps and per third of the scheduler-phase range.

Matched-budget factorization (Sec. 5.4): placement (risk controller vs
periodic) crossed with construction (lifted surrogate vs native latent
secant) at the same number of exact calls, scored by the final latent's
distance to the all-exact rollout.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from . import _binding as B


# ---------------------------------------------------------------- statistics

def pearson(x, y) -> float:
    x, y = np.asarray(x, np.float64), np.asarray(y, np.float64)
    if len(x) < 2:
        return float("nan")
    xc, yc = x - x.mean(), y - y.mean()
    den = np.sqrt((xc * xc).sum() * (yc * yc).sum())
    return float((xc * yc).sum() / den) if den > 0 else float("nan")


def ranks(x) -> np.ndarray:
    """1-based ranks, ties sharing their average rank."""
    x = np.asarray(x, np.float64)
    order = np.argsort(x, kind="mergesort")
    r = np.empty(len(x))
    i = 0
    while i < len(x):
        j = i
        while j + 1 < len(x) and x[order[j + 1]] == x[order[i]]:
            j += 1
        r[order[i:j + 1]] = (i + j) / 2.0 + 1.0
        i = j + 1
    return r


def spearman(x, y) -> float:
    return pearson(ranks(x), ranks(y))


def false_safe(criterion, down, phase, bins: int = 3) -> Dict[str, float]:
    """Share of steps deemed safe (criterion <= its median) whose downstream
    degradation exceeds the median degradation; overall and per phase bin
    (bin b holds phases in [b/bins, (b+1)/bins), the last bin closed)."""
    c, d, q = (np.asarray(a, np.float64) for a in (criterion, down, phase))
    if len(c) == 0:
        return {"all": float("nan")}
    safe = c <= np.median(c)
    bad = d > np.median(d)
    out = {"all": float((safe & bad).sum() / max(safe.sum(), 1))}
    b = np.minimum((q * bins).astype(np.int64), bins - 1)
    for i in range(bins):
        m = safe & (b == i)
        out[f"phase_bin{i}"] = float((m & bad).sum() / m.sum()) if m.any() else float("nan")
    return out


def l1_rel(a, b, eps: float = 1e-8) -> float:
    """mean|a - b| / (mean|b| + eps), the normalisation of Eq. (7)."""
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.mean(np.abs(a - b)) / (np.mean(np.abs(b)) + eps))


def l2_rel(a, b) -> float:
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


# ---------------------------------------------------------------- rollouts

@dataclass
class Inputs:
    """Device tensors of one rollout's conditioning; replay_v replaces F_theta."""
    z_T: object
    cond: object = None
    text: object = None
    cam: object = None
    replay_v: object = None


def _run(ctx: "B.Context", state, inp: Inputs, steps: int, mode: int, forced=None):
    z = inp.z_T.clone()
    sched, logs = ctx.rollout(state, z, steps, inp.cond, inp.text, inp.cam, mode=mode, forced=forced,
                              replay_v=inp.replay_v)
    return z, sched, logs


@dataclass
class Sweep:
    phase: List[float] = field(default_factory=list)      # q_t of each injected step
    step: List[int] = field(default_factory=list)
    d_local: List[float] = field(default_factory=list)    # d_t
    d_hat: List[float] = field(default_factory=list)
    delta: List[float] = field(default_factory=list)      # w_t * d_hat_t
    down: List[float] = field(default_factory=list)       # D_t^down
    anchor_d_hat: List[float] = field(default_factory=list)
    anchor_d_cf: List[float] = field(default_factory=list)

    def extend(self, o: "Sweep"):
        for k in self.__dataclass_fields__:
            getattr(self, k).extend(getattr(o, k))

    def summary(self) -> dict:
        return {
            "injections": len(self.step),
            "pearson_dhat_dcf": pearson(self.anchor_d_hat, self.anchor_d_cf),
            "spearman_dhat_dcf": spearman(self.anchor_d_hat, self.anchor_d_cf),
            "pearson_down_local": pearson(self.d_hat, self.down),
            "spearman_down_local": spearman(self.d_hat, self.down),
            "pearson_down_weighted": pearson(self.delta, self.down),
            "spearman_down_weighted": spearman(self.delta, self.down),
            "false_safe_local_defect": false_safe(self.d_local, self.down, self.phase),
            "false_safe_weighted_risk": false_safe(self.delta, self.down, self.phase),
        }


def injection_sweep(ctx: "B.Context", inp: Inputs, steps: int, eps: float = 1e-8) -> Sweep:
    """One all-exact rollout, then one rollout per step t >= 1 with the
    surrogate forced at t only (skipped where the candidate is unavailable)."""
    st = ctx.new_state()
    z_ref, sched, logs = _run(ctx, st, inp, steps, B.MODE_ALL_EXACT)
    assert sched == [0] * steps
    ref = z_ref.float().cpu().numpy()
    out = Sweep()
    for g in logs:
        if np.isfinite(g["d_cf"]):
            out.anchor_d_hat.append(g["d_hat"])
            out.anchor_d_cf.append(g["d_cf"])
    for t in range(1, steps):
        if not logs[t]["available"]:
            continue
        mask = [0] * steps
        mask[t] = 1
        z, s, lg = _run(ctx, st, inp, steps, B.MODE_FORCED, forced=mask)
        assert s == mask
        out.step.append(t)
        out.phase.append(lg[t]["t"])
        out.d_local.append(logs[t]["d_cf"])
        out.d_hat.append(lg[t]["d_hat"])
        out.delta.append(lg[t]["w"] * lg[t]["d_hat"])
        out.down.append(l1_rel(z.float().cpu().numpy(), ref, eps))
    return out


def _share_weights(ctx: "B.Context", src: "B.Context"):
    ctx.weights = src.weights
    if src.weights is not None:
        ctx._check(ctx.lib.wdc_bind_weights(ctx.h, B.C.c_void_p(src.weights.data_ptr()), src.weights.numel()))


def variant_context(src: "B.Context", **params) -> "B.Context":
    """A context for the same model (weights shared with ``src``) with other parameters."""
    p = B.default_params()
    for f, _ in B.Params._fields_:
        setattr(p, f, getattr(src.params, f))
    for k, v in params.items():
        setattr(p, k, v)
    ctx = B.Context(src.cfg, params=p, device=str(src.device), allocate_weights=False)
    _share_weights(ctx, src)
    return ctx


def risk_threshold_for_budget(ctx_of, inp: Inputs, steps: int, n_exact: int, lo: float = 0.0,
                              hi: float = 8.0, iters: int = 40):
    """Bisection on tau_risk for a risk-controlled rollout with ``n_exact`` exact
    calls (the count falls as tau grows). ``ctx_of(tau)`` returns a context.
    Returns (tau, schedule, z) of the closest count found."""
    best = None
    for _ in range(iters):
        tau = 0.5 * (lo + hi)
        ctx = ctx_of(tau)
        z, sched, _ = _run(ctx, ctx.new_state(), inp, steps, B.MODE_RISK)
        n = steps - sum(sched)
        if best is None or abs(n - n_exact) < abs(best[1] - n_exact):
            best = (tau, n, sched, z)
        if n == n_exact:
            break
        if n > n_exact:
            lo = tau
        else:
            hi = tau
    return best[0], best[2], best[3]


def factorization(ctx: "B.Context", inp: Inputs, steps: int, period: int) -> Dict[str, dict]:
    """Periodic / risk placement x lifted / secant construction at the exact-call
    budget of periodic placement with ``period``; final-latent distance to the
    all-exact rollout."""
    z_ref, _, _ = _run(ctx, ctx.new_state(), inp, steps, B.MODE_ALL_EXACT)
    ref = z_ref.float().cpu().numpy()
    n_exact = len(range(0, steps, period))
    out = {}
    for cons, code in (("lifted", B.SURROGATE_LIFTED), ("secant", B.SURROGATE_SECANT)):
        pc = variant_context(ctx, surrogate=code, period=period)
        t0 = time.perf_counter()
        z, sched, _ = _run(pc, pc.new_state(), inp, steps, B.MODE_PERIODIC)
        dt = time.perf_counter() - t0
        zz = z.float().cpu().numpy()
        out[f"periodic+{cons}"] = {"exact_calls": steps - sum(sched), "l1_rel": l1_rel(zz, ref),
                                   "l2_rel": l2_rel(zz, ref), "seconds": dt}
        tau, sched, z = risk_threshold_for_budget(
            lambda tau: variant_context(ctx, surrogate=code, tau_risk=tau), inp, steps, n_exact)
        zz = z.float().cpu().numpy()
        out[f"risk+{cons}"] = {"exact_calls": steps - sum(sched), "tau_risk": tau, "l1_rel": l1_rel(zz, ref),
                               "l2_rel": l2_rel(zz, ref)}
    return out


def main(argv=None):
    """Diagnostics on a synthetic workload with device random-init weights;
    prints one JSON object."""
    import argparse
    import dataclasses
    import json

    import torch

    import synth

    ap = argparse.ArgumentParser(description=main.__doc__)
    ap.add_argument("--workload", default="mid", choices=["tiny", "mid", "5b"])
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--seeds", type=int, default=4)
    ap.add_argument("--period", type=int, default=4)
    a = ap.parse_args(argv)
    cfg = synth.get_config(a.workload)
    ctx = B.Context(cfg)
    ctx.init_random_weights(seed=1234, std=0.02)
    sweep = Sweep()
    t0 = time.perf_counter()
    fact = None
    for s in range(a.seeds):
        c = dataclasses.replace(cfg, seed=cfg.seed + 100 * s)
        inp = synth.gen_inputs(c)
        dev = {k: (ctx.to_device(v, dtype=torch.float32) if k == "z_T" else ctx.to_device(v))
               for k, v in inp.items()}
        gin = Inputs(dev["z_T"], dev.get("cond"), dev.get("text"), dev.get("cam"))
        sweep.extend(injection_sweep(ctx, gin, a.steps))
        if s == 0:
            fact = factorization(ctx, gin, a.steps, a.period)
    torch.cuda.synchronize()
    out = {"workload": a.workload, "steps": a.steps, "seeds": a.seeds, "seconds": round(time.perf_counter() - t0, 2),
           "injection": sweep.summary(), "factorization": fact}
    print(json.dumps(out, default=float))


if __name__ == "__main__":
    main()
