"""GPU parity of the controller and surrogate variants of the ablation study
(Sec. 5.4, matched-budget tables) against the oracle: periodic placement, the
native latent secant, linear observation, the lift without condition, and the
controller switches. Recorded velocities stand in for F_theta (replay rollouts)
except in the last test, which runs the tiny DiT. Schedules must match bit for
bit (thresholds chosen with clear oracle margins); latents within the float32
tolerance."""
from dataclasses import replace

import numpy as np
import pytest

import synth
from oracle import params as P
from oracle import rollout as ro
from tests.gpu_util import TOL_F32, context, dev_inputs, pick_tau, rel_l2, torch_cuda, wdc_params

pytestmark = pytest.mark.gpu

MODES = {"risk": 0, "forced": 1, "all_exact": 2, "periodic": 3}

# name: (oracle parameter overrides, mode)
VARIANTS = {
    "periodic_lifted": (dict(period=4), "periodic"),
    "periodic_secant": (dict(period=4, surrogate="secant"), "periodic"),
    "risk_secant": (dict(surrogate="secant"), "risk"),
    "risk_linear_observation": (dict(observation="linear"), "risk"),
    "periodic_linear_observation": (dict(observation="linear", period=3), "periodic"),
    "instantaneous_risk": (dict(lam=0.0), "risk"),
    "no_impact_weighting": (dict(impact_weight=False), "risk"),
    "no_calibration": (dict(calibrate=False), "risk"),
}


def compare(glogs, ologs, tol=1e-4):
    for g, o in zip(glogs, ologs):
        assert g["exact"] == int(o.exact) and g["bank"] == o.bank
        assert g["support"] == o.support and g["available"] == int(o.available)
        for key in ("d_z", "p", "w", "r_cand", "eta", "R", "alpha"):
            a, b = g[key], getattr(o, key)
            assert abs(a - b) <= tol * max(1.0, abs(b)), (o.k, key, a, b)
        if np.isfinite(o.d_cf):
            assert abs(g["d_cf"] - o.d_cf) <= tol * max(1.0, o.d_cf), (o.k, g["d_cf"], o.d_cf)
        else:
            assert not np.isfinite(g["d_cf"])
        if o.bank:
            np.testing.assert_allclose(g["pi"], o.pi, atol=10 * tol)
            np.testing.assert_allclose(g["kappa"], o.kappa, atol=10 * tol)
            np.testing.assert_allclose(g["sims_in"], o.sims_in, atol=tol)


def run_variant(cfg, steps, overrides, mode, forced=None, target=None, cam=None):
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    vel = synth.gen_replay_velocities(cfg, steps)
    z0 = synth.gen_inputs(cfg)["z_T"]
    den = ro.replay_denoiser(vel)
    base = P.with_(P.DEFAULTS, **overrides)
    if mode == "risk":
        tau, ref = pick_tau(lambda tau: ro.rollout(den, z0, steps, P.with_(base, tau_risk=tau), cam=cam),
                            lo=0.05, hi=1.5, target_surrogates=target or steps // 2)
        base = P.with_(base, tau_risk=tau)
    else:
        ref = ro.rollout(den, z0, steps, base, mode=mode, forced=forced, cam=cam)
    ctx = context(cfg, weights=False, params=wdc_params(base))
    z = torch.from_numpy(z0).cuda()
    camd = ctx.to_device(cam) if cam is not None else None
    sched, logs = ctx.rollout(ctx.new_state(), z, steps, cam=camd, mode=MODES[mode], forced=forced,
                              replay_v=torch.from_numpy(vel).cuda())
    print(cfg.name, overrides, mode, "schedule", sched)
    assert sched == ref.schedule
    compare(logs, ref.log)
    err = rel_l2(z.cpu().numpy(), ref.z)
    print("final latent rel_l2", err)
    assert err <= TOL_F32
    return ref


@pytest.mark.parametrize("name", list(VARIANTS))
def test_variant_tiny_latent_20_steps(name):
    overrides, mode = VARIANTS[name]
    ref = run_variant(synth.get_config("tiny"), 20, overrides, mode)
    if mode == "periodic":
        assert all(ref.schedule[k] == 0 for k in range(0, 20, overrides["period"]))


@pytest.mark.parametrize("name", ["periodic_secant", "risk_linear_observation", "no_impact_weighting"])
def test_variant_mid_latent(name):
    overrides, mode = VARIANTS[name]
    run_variant(synth.get_config("mid"), 20, overrides, mode)


def test_no_support_constraint_commits_unsupported_candidates():
    mask = [0, 1, 1, 0, 1, 1, 0, 1]
    ref = run_variant(synth.get_config("tiny"), 8, dict(theta_sim=1.5, support_constraint=False), "forced",
                      forced=mask)
    assert ref.schedule == mask and all(l.support == 0 for l in ref.log)


def test_lift_without_condition_with_camera():
    """A camera vector enters the summary and retrieval only when condition is on."""
    cfg = replace(synth.get_config("tiny"), name="tiny_cam", cam_dim=48)
    cam = synth.gen_inputs(cfg)["cam"]
    run_variant(cfg, 20, dict(lift_condition=False), "risk", cam=cam)
    run_variant(cfg, 20, dict(), "risk", cam=cam)


@pytest.mark.parametrize("overrides", [dict(surrogate="secant"), dict(observation="linear")])
def test_variant_largest_latent_forced(overrides):
    """16 x 33 x 90 x 160 latent; 4 exact inserts fill the bank (and its input latents)."""
    mask = [0, 1, 0, 0, 1, 0, 1, 1]
    run_variant(synth.get_config("stress"), 8, dict(overrides, theta_sim=-1.0), "forced", forced=mask)


def test_periodic_secant_tiny_dit_matches_oracle():
    """F_theta evaluated (tiny float32 DiT) with periodic placement and the secant."""
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    cfg = synth.get_config("tiny")
    W = synth.gen_weights(cfg)
    inp = synth.gen_inputs(cfg)
    p = P.with_(P.DEFAULTS, period=3, surrogate="secant")
    ref = ro.rollout(ro.dit_denoiser(W, cfg, inp), inp["z_T"], 8, p, mode="periodic")
    ctx = context(cfg, params=wdc_params(p))
    _, dv = dev_inputs(ctx, cfg)
    z = dv["z_T"].clone()
    sched, logs = ctx.rollout(ctx.new_state(), z, 8, dv["cond"], mode=wdc.MODE_PERIODIC)
    assert sched == ref.schedule == [0, 1, 1, 0, 1, 1, 0, 1]
    compare(logs, ref.log)
    assert rel_l2(z.cpu().numpy(), ref.z) <= TOL_F32


@pytest.mark.parametrize("capacity", [1, 8])
def test_bank_capacity_extremes(capacity):
    """FIFO of one record (every insert replaces it) and of the largest capacity the
    kernels take; 30 steps so the 8-slot bank wraps around."""
    mode = "forced"
    mask = [0 if k % 3 == 0 else 1 for k in range(30)]
    run_variant(synth.get_config("tiny"), 30, dict(bank_capacity=capacity, theta_sim=-1.0), mode, forced=mask)


@pytest.mark.parametrize("steps", [1, 2])
def test_shortest_rollouts(steps):
    """One step (always exact: empty bank) and two steps (the second may commit a
    candidate built from a single record)."""
    ref = run_variant(synth.get_config("tiny"), steps, dict(tau_risk=float("inf")), "forced",
                      forced=[1] * steps)
    assert ref.schedule[0] == 0


def test_open_threshold_takes_every_available_step():
    ref = run_variant(synth.get_config("tiny"), 20, dict(tau_risk=1e9, theta_sim=-1.0), "forced",
                      forced=[1] * 20)
    assert ref.schedule == [0 if k % 8 == 0 else 1 for k in range(20)]
