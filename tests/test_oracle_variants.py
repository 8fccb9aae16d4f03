"""Pins for the controller and surrogate variants of the ablation study
(Sec. 5.4, matched-budget tables) in the oracle, CPU only: periodic placement,
the native latent secant, linear observation, the lift without condition, and
the controller switches (instantaneous risk, no impact weighting, no
counterfactual calibration, no support constraint)."""
import numpy as np
import pytest

import synth
from oracle import params as P
from oracle import risk as rk
from oracle import rollout as ro
from oracle import surrogate as sg

PR = P.DEFAULTS
CFG = synth.get_config("tiny")
SHAPE = (16, 2, 4, 6)


def replay(steps):
    return ro.replay_denoiser(synth.gen_replay_velocities(CFG, steps))


def z0():
    return synth.gen_inputs(CFG)["z_T"]


# --------------------------------------------------------------------------- periodic placement

@pytest.mark.parametrize("period,S", [(4, 20), (3, 8), (8, 50)])
def test_periodic_schedule_closed_form(period, S):
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, period=period), mode="periodic")
    assert res.schedule == [0 if k % period == 0 else 1 for k in range(S)]
    assert res.calls == len(range(0, S, period))


def test_periodic_one_is_all_exact_bitwise():
    S = 8
    a = ro.rollout(replay(S), z0(), S, P.with_(PR, period=1), mode="periodic")
    b = ro.rollout(replay(S), z0(), S, PR, mode="all_exact")
    assert a.schedule == [0] * S
    np.testing.assert_array_equal(a.z, b.z)


def test_periodic_placement_ignores_risk_threshold():
    S = 20
    lo = ro.rollout(replay(S), z0(), S, P.with_(PR, period=4, tau_risk=-1.0), mode="periodic")
    hi = ro.rollout(replay(S), z0(), S, P.with_(PR, period=4, tau_risk=1e9), mode="periodic")
    assert lo.schedule == hi.schedule
    np.testing.assert_array_equal(lo.z, hi.z)


# --------------------------------------------------------------------------- native latent secant

def test_secant_reuses_latest_exact_increment():
    """Psi is the Euler step, so the latest exact transition is z_a -> z_a + dt*v_a:
    on the uniform grid every secant step adds dt * v_a of the latest exact step a."""
    S = 12
    vel = synth.gen_replay_velocities(CFG, S)
    trace = []
    p = P.with_(PR, surrogate="secant", period=4)
    res = ro.rollout(ro.replay_denoiser(vel), z0(), S, p, mode="periodic", trace=trace)
    assert res.schedule == [0 if k % 4 == 0 else 1 for k in range(S)]
    z_prev = np.asarray(z0(), np.float64)
    for k in range(S):
        a = 4 * (k // 4)
        np.testing.assert_allclose(trace[k] - z_prev, -vel[a].astype(np.float64) / S, atol=1e-12)
        z_prev = trace[k]


def test_secant_exact_for_constant_velocity():
    S = 16
    v = synth.gen_replay_velocities(CFG, 1)[0]
    const = ro.replay_denoiser(np.stack([v] * S))
    p = P.with_(PR, surrogate="secant", tau_risk=np.inf)
    res = ro.rollout(const, z0(), S, p)
    assert sum(res.schedule) > S // 2
    np.testing.assert_allclose(res.z, np.asarray(z0(), np.float64) - v, atol=1e-12)
    dcf = [l.d_cf for l in res.log if np.isfinite(l.d_cf)]
    assert dcf and max(dcf) < 1e-12


def test_secant_unavailable_before_first_exact_and_logs():
    bank = sg.Bank(4)
    assert sg.secant_candidate(np.ones(SHAPE), None, bank, 1.0, 0.9, 0.0, 0.0, PR) is None
    S = 8
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, surrogate="secant", period=2), mode="periodic")
    for l in res.log[1:]:
        assert l.support == 1 and l.alpha == pytest.approx(1.0, rel=1e-12)
        assert sum(l.pi) == 1.0 and sum(l.kappa) == 0.0


# --------------------------------------------------------------------------- linear observation

def rms_equal_bank(rng, q0=0.8, dq=0.05):
    """A one-record bank whose latents are permutations of one vector (equal RMS)."""
    x = rng.standard_normal(int(np.prod(SHAPE)))
    z_in, z_out, z_cur = (rng.permutation(x).reshape(SHAPE) for _ in range(3))
    bank = sg.Bank(4)
    cam = np.zeros(16)
    pin, pout = sg.lift(z_in, None, None, q0, cam, PR), sg.lift(z_out, None, None, q0 - dq, cam, PR)
    bank.insert(sg.Record(pin, pout, sg.summary(pin), sg.summary(pout), q0, q0 - dq, z_out))
    return bank, z_in, z_out, z_cur


def test_linear_readout_equal_rms_closed_form():
    """With equal RMS the normalisation cancels and the lifted step reads back as
    z_t + alpha * (z_out - z_in); on the uniform grid alpha = dt/(dt + eps)."""
    rng = np.random.default_rng(3)
    bank, z_in, z_out, z_cur = rms_equal_bank(rng)
    p = P.with_(PR, observation="linear", theta_sim=-1.0)
    phi = sg.lift(z_cur, z_in, None, 0.75, np.zeros(16), p)
    c = sg.candidate(phi, bank, 0.70, 0.8, 0.75, p, z=z_cur)
    assert c.support == [0] and c.pi.tolist() == [1.0]
    alpha = 0.05 / (0.05 + p.eps)
    np.testing.assert_allclose(c.z_hat, z_cur + alpha * (z_out - z_in), atol=1e-12)
    assert c.kappa.tolist() == [0.0]


def test_linear_readout_empty_support_returns_current_latent():
    rng = np.random.default_rng(4)
    bank, z_in, z_out, z_cur = rms_equal_bank(rng)
    p = P.with_(PR, observation="linear", theta_sim=1.5)
    phi = sg.lift(z_cur, z_in, None, 0.75, np.zeros(16), p)
    c = sg.candidate(phi, bank, 0.70, 0.8, 0.75, p, z=z_cur)
    assert c.support == []
    np.testing.assert_allclose(c.z_hat, z_cur, rtol=1e-14, atol=1e-14)


def test_linear_readout_is_positively_homogeneous():
    rng = np.random.default_rng(5)
    z_in, z_out, z_cur = (rng.standard_normal(SHAPE) for _ in range(3))
    p = P.with_(PR, observation="linear", theta_sim=-1.0, eps_nu=0.0)

    def cand(scale):
        bank = sg.Bank(4)
        pin = sg.lift(scale * z_in, None, None, 0.8, np.zeros(16), p)
        pout = sg.lift(scale * z_out, None, None, 0.75, np.zeros(16), p)
        bank.insert(sg.Record(pin, pout, sg.summary(pin), sg.summary(pout), 0.8, 0.75, scale * z_out))
        phi = sg.lift(scale * z_cur, scale * z_in, None, 0.75, np.zeros(16), p)
        return sg.candidate(phi, bank, 0.70, 0.8, 0.75, p, z=scale * z_cur).z_hat

    np.testing.assert_allclose(cand(3.0), 3.0 * cand(1.0), rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------- lift without condition

def test_no_condition_lift_ignores_camera_and_phase():
    rng = np.random.default_rng(6)
    base = rng.standard_normal(SHAPE)
    cam_a = sg.cam_descriptor(rng.standard_normal(48), PR.eps_nu)
    cam_b = sg.cam_descriptor(rng.standard_normal(48), PR.eps_nu)
    z_in, z_out = base, base + 0.05 * rng.standard_normal(SHAPE)
    z = z_out + 0.01 * rng.standard_normal(SHAPE)

    def cand(p, cam, q_in):
        bank = sg.Bank(4)
        pin, pout = sg.lift(z_in, None, None, q_in, cam, p), sg.lift(z_out, None, None, q_in - 0.05, cam, p)
        bank.insert(sg.Record(pin, pout, sg.summary(pin), sg.summary(pout), q_in, q_in - 0.05, z_out))
        phi = sg.lift(z, z_in, None, 0.3, cam_a, p)
        return sg.candidate(phi, bank, 0.25, q_in, q_in - 0.05, p, z=z)

    off = P.with_(PR, lift_condition=False)
    # q_in = 0.9 lies beyond theta_q from q = 0.3: excluded only when phase is used
    c1, c2 = cand(off, cam_a, 0.9), cand(off, cam_b, 0.35)
    assert c1.support == [0] and c2.support == [0]
    np.testing.assert_array_equal(c1.sims_in, c2.sims_in)
    np.testing.assert_array_equal(sg.summary(sg.lift(z, z_in, None, 0.3, cam_b, off))[224:240], 0)
    on = cand(PR, cam_a, 0.9)
    assert on.support == []


# --------------------------------------------------------------------------- controller switches

def test_instantaneous_risk_is_the_current_increment():
    S = 20
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, lam=0.0, tau_risk=0.3))
    for l in res.log:
        assert l.r_cand == pytest.approx(l.w * l.d_hat, rel=1e-15)
        assert l.R == (l.r_cand if not l.exact else 0.0)


def test_no_impact_weighting_sets_w_to_one():
    assert rk.sensitivity_weight(1.0, P.with_(PR, impact_weight=False), 5.0, 5.0) == 1.0
    S = 20
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, impact_weight=False, tau_risk=0.3))
    assert all(l.w == 1.0 for l in res.log)
    full = ro.rollout(replay(S), z0(), S, P.with_(PR, tau_risk=0.3))
    assert any(l.w > 1.0 for l in full.log)


def test_frozen_calibration_keeps_eta():
    S = 20
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, calibrate=False, tau_risk=0.3))
    assert any(np.isfinite(l.d_cf) for l in res.log)
    assert all(l.eta == PR.eta0 for l in res.log)


def test_no_support_constraint_commits_unsupported_candidates():
    S = 8
    mask = [0, 1, 1, 0, 1, 1, 0, 1]
    closed = P.with_(PR, theta_sim=1.5)       # nothing is ever in N_t
    on = ro.rollout(replay(S), z0(), S, closed, mode="forced", forced=mask)
    off = ro.rollout(replay(S), z0(), S, P.with_(closed, support_constraint=False), mode="forced", forced=mask)
    assert on.schedule == [0] * S
    assert off.schedule == mask
    assert all(l.support == 0 for l in off.log)
    # the counterfactual is still taken on exact steps with a finite candidate
    assert any(np.isfinite(l.d_cf) for l in off.log)
