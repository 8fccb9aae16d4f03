"""Write the oracle's threshold sweeps used by the rollout parity tests.

Calls only the oracle (and the seeded inputs). Two kinds of sweep:

* ``--kind dit --workload mid``: rollouts that evaluate the synthetic F_theta,
  thresholds giving 0, 2, ..., 12 surrogate steps of 20 (0-60% skipped).
  Every visited schedule is saved with its threshold interval, per-step
  controller log, the final latent at fixed sampled positions and its full
  L2 norm; ``--kind select`` keeps the widest-margin schedule for each count,
  so the GPU test needs no oracle F_theta at run time.
* ``--kind replay --workload 5b|13b``: rollouts on recorded velocities at the
  workload's latent, thresholds giving the exact-call ratios of the paper's
  world-generation settings (Sec. 5.1: 47% for the 5B model, 20% for the 13B
  model, from exact_ratio_targets.json). Only thresholds and schedules are
  saved; the test re-runs the oracle.

Usage:
  python tests/golden/make_tau_sweeps.py --kind dit --workload mid --out /tmp/mid_full
  python tests/golden/make_tau_sweeps.py --kind select --select /tmp/mid_full.json --out tests/golden/mid_tau_sweep
  python tests/golden/make_tau_sweeps.py --kind replay --workload 13b --out tests/golden/replay_thresholds
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import synth  # noqa: E402
from oracle import params as P  # noqa: E402
from oracle import rollout as ro  # noqa: E402
from tests import tau_search as ts  # noqa: E402

LOG_KEYS = ("exact", "bank", "support", "available", "finite", "d_z", "p", "d_hat", "w", "r_cand", "eta", "R",
            "alpha", "sim_margin")
N_SAMPLES = 2048


def log(msg):
    print(f"[sweep {time.strftime('%H:%M:%S')}] {msg}", flush=True)


def sample_index(numel: int, seed: int = 20250) -> np.ndarray:
    return np.sort(np.random.default_rng(seed).choice(numel, size=min(N_SAMPLES, numel), replace=False))


def dit_sweep(args):
    cfg = synth.get_config(args.workload)
    S = args.steps or cfg.steps
    W = synth.gen_weights(cfg)
    inp = synth.gen_inputs(cfg)
    cache = {}
    den = ts.memo_denoiser(ro.dit_denoiser(W, cfg, inp), cache)
    idx = sample_index(cfg.numel)
    records = json.load(open(args.resume))["schedules"] if args.resume else []

    def run(tau):
        t0 = time.time()
        res = ro.rollout(den, inp["z_T"], S, P.with_(P.DEFAULTS, tau_risk=tau), cam=inp.get("cam"))
        a, b = ts.interval(res)
        records.append({"interval": [a, b if math.isfinite(b) else None], "schedule": res.schedule,
                        "log": [{k: float(getattr(l, k)) for k in LOG_KEYS} for l in res.log],
                        "kappa": [list(map(float, l.kappa)) for l in res.log],
                        "final_norm": float(np.linalg.norm(res.z)),
                        "final_samples": res.z.reshape(-1)[idx].tolist()})
        save(args, cfg, S, idx, records)
        log(f"rollout {len(records)}: {sum(res.schedule)} surrogate steps, interval [{a:.6g}, {b:.6g}), "
            f"{len(cache)} F_theta evaluations so far, {time.time() - t0:.1f}s")
        return res

    targets = tuple(range(0, 13, 2))
    t_start = time.time()

    def timed_run(tau):
        if time.time() - t_start > args.max_seconds:
            raise TimeoutError
        return run(tau)
    try:
        ts.explore(timed_run, lo=args.lo, hi=args.hi, budget=args.budget, targets=targets,
                   min_margin=args.min_margin, known=_seen(records))
    except TimeoutError:
        log(f"stopped after {args.max_seconds} s; {len(records)} schedules saved")
    for n in targets:
        log(f"{n} surrogate steps: tau, margin = {ts.pick(_seen(records), n)}")


def _seen(records):
    return [(r["interval"][0], math.inf if r["interval"][1] is None else r["interval"][1], sum(r["schedule"]),
             r["schedule"]) for r in records]


def save(args, cfg, S, idx, records):
    out = {"workload": cfg.name, "steps": S, "sample_index": idx.tolist(), "schedules": records,
           "note": "written by tests/golden/make_tau_sweeps.py from the oracle alone"}
    with open(args.out + ".json", "w") as f:
        json.dump(out, f)


def select(args):
    """Keep, for each wanted count of surrogate steps, the saved schedule with the
    widest margin, and put its threshold at the centre of its interval."""
    full = json.load(open(args.select))
    seen = _seen(full["schedules"])
    keep = []
    for n in range(0, 13, 2):
        tau, m = ts.pick(seen, n)
        if not m > 0:
            log(f"no schedule with {n} surrogate steps")
            continue
        rec = next(r for r, (a, b, c, _) in zip(full["schedules"], seen)
                   if c == n and abs(ts.centre(a, b) - tau) <= 1e-15 * max(1.0, tau))
        keep.append(dict(rec, tau=tau, margin=m))
        log(f"{n} surrogate steps: tau {tau:.6g}, margin {m:.3g}")
    out = {k: v for k, v in full.items() if k != "schedules"}
    out["cases"] = keep
    with open(args.out + ".json", "w") as f:
        json.dump(out, f)


def replay_sweep(args):
    cfg = synth.get_config(args.workload)
    S = args.steps or cfg.steps
    targets = json.load(open(os.path.join(HERE, "exact_ratio_targets.json")))
    ratio = targets["aether_5b" if args.workload == "5b" else "voyager_13b"]
    n_exact = ratio * S
    want = sorted({S - math.floor(n_exact), S - math.ceil(n_exact)})
    vel = synth.gen_replay_velocities(cfg, S)
    z0 = synth.gen_inputs(cfg)["z_T"]
    den = ro.replay_denoiser(vel)

    def run(tau):
        t0 = time.time()
        res = ro.rollout(den, z0, S, P.with_(P.DEFAULTS, tau_risk=tau))
        log(f"tau {tau:.6g}: {sum(res.schedule)} surrogate steps ({time.time() - t0:.1f}s)")
        return res

    seen = ts.explore(run, lo=args.lo, hi=args.hi, budget=args.budget, targets=want, min_margin=args.min_margin)
    best = max(((n, *ts.pick(seen, n)) for n in want), key=lambda x: x[2])
    n, tau, m = best
    sched = next(s for a, b, c, s in seen if c == n and abs(ts.centre(a, b) - tau) < 1e-15 * max(1.0, tau))
    entry = {"workload": cfg.name, "steps": S, "target_exact_ratio": ratio, "tau": tau, "margin": m,
             "surrogate_steps": n, "exact_calls": S - n, "schedule": sched,
             "note": "written by tests/golden/make_tau_sweeps.py from the oracle alone"}
    path = args.out + ".json"
    allj = json.load(open(path)) if os.path.exists(path) else {}
    allj[cfg.name] = entry
    with open(path, "w") as f:
        json.dump(allj, f, indent=1)
    log(f"{cfg.name}: tau {tau:.6g}, {S - n} exact of {S}, margin {m:.3g}")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--kind", choices=["dit", "replay", "select"], required=True)
    ap.add_argument("--workload", default="mid")
    ap.add_argument("--select", help="with --kind select: a full dit sweep file to pick the test cases from")
    ap.add_argument("--steps", type=int, default=0)
    ap.add_argument("--out", required=True)
    ap.add_argument("--lo", type=float, default=1e-3)
    ap.add_argument("--hi", type=float, default=10.0)
    ap.add_argument("--budget", type=int, default=60)
    ap.add_argument("--min-margin", type=float, default=0.03)
    ap.add_argument("--max-seconds", type=float, default=math.inf)
    ap.add_argument("--resume", help="with --kind dit: a full sweep file whose schedules are kept and not re-run")
    args = ap.parse_args()
    {"dit": dit_sweep, "replay": replay_sweep, "select": select}[args.kind](args)


if __name__ == "__main__":
    main()
