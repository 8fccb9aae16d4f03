"""Pins for the oracle scheduler and inference loop (Eq. (1), Sec. 4.3-4.4), CPU only."""
import json
import os

import numpy as np
import pytest

import synth
from oracle import params as P
from oracle import rollout as ro
from oracle import scheduler as sch

HERE = os.path.dirname(__file__)
PR = P.DEFAULTS
CFG = synth.get_config("tiny")


def replay(steps):
    return ro.replay_denoiser(synth.gen_replay_velocities(CFG, steps))


def z0():
    return synth.gen_inputs(CFG)["z_T"]


# --------------------------------------------------------------------------- Psi

def test_psi_constant_velocity_closed_form():
    rng = np.random.default_rng(0)
    z_start, c = rng.standard_normal((4, 5)), rng.standard_normal((4, 5))
    S = 20
    z = z_start
    for k in range(S):
        z = sch.psi(z, c, sch.t_at(k, S), sch.t_at(k + 1, S))
    # the steps dt sum to t_S - t_0 = -1
    np.testing.assert_allclose(z, z_start - c, atol=1e-12)


def test_psi_linear_velocity_closed_form():
    lam, S = -0.7, 16
    z = np.ones(3)
    for k in range(S):
        z = sch.psi(z, lam * z, sch.t_at(k, S), sch.t_at(k + 1, S))
    np.testing.assert_allclose(z, np.prod([1 - lam / S for _ in range(S)]) * np.ones(3), rtol=1e-13)


def test_time_grid():
    g = sch.time_grid(8)
    assert g[0] == 1.0 and g[-1] == 0.0 and len(g) == 9
    np.testing.assert_allclose(np.diff(g), -1 / 8)


# --------------------------------------------------------------------------- schedules

def test_age_limit_reproduces_paper_exact_ratio():
    gold = json.load(open(os.path.join(HERE, "golden", "paper_schedule.json")))
    S = gold["steps"]
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, tau_risk=np.inf))
    exact = [k for k, s in enumerate(res.schedule) if s == 0]
    assert exact == gold["exact_steps"]
    assert len(exact) == gold["exact_calls"]
    assert len(exact) / S == pytest.approx(gold["exact_ratio"])
    assert res.calls == len(exact) == res.inserts


@pytest.mark.parametrize("S,expect", [(20, [0, 8, 16]), (8, [0, 4])])
def test_open_threshold_schedules(S, expect):
    """S=20: the age limit alone (8 x 1/20 = 0.4 <= theta_q). S=8: after 4 steps of 1/8
    the only record's phase is 0.5 away (> theta_q = 0.43), so support runs out first."""
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, tau_risk=np.inf))
    assert [k for k, s in enumerate(res.schedule) if s == 0] == expect


def test_all_exact_equals_plain_euler_bitwise():
    S = 8
    den = replay(S)
    res = ro.rollout(den, z0(), S, PR, mode="all_exact")
    z = np.asarray(z0(), dtype=np.float64)
    for k in range(S):
        z = sch.psi(z, den(z, k, sch.t_at(k, S)), sch.t_at(k, S), sch.t_at(k + 1, S))
    assert res.schedule == [0] * S
    np.testing.assert_array_equal(res.z, z)
    assert res.calls == S and res.inserts == S


def test_calls_and_inserts_equal_exact_steps_and_fifo():
    S = 20
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, tau_risk=0.35))
    n_exact = res.schedule.count(0)
    assert 0 < n_exact < S
    assert res.calls == n_exact == res.inserts
    slots = [l.slot for l in res.log if l.exact]
    assert slots == [i % PR.bank_capacity for i in range(n_exact)]
    assert all(l.slot == -1 for l in res.log if not l.exact)
    # risk bookkeeping: after a surrogate R = R_cand, after an exact step R = lambda * R_prev
    R = PR.r0
    for l in res.log:
        R = l.r_cand if not l.exact else PR.lam * R
        assert l.R == pytest.approx(R, rel=1e-12)
        assert l.margin >= 0


def test_counterfactual_calibration_happens_only_with_support():
    S = 20
    res = ro.rollout(replay(S), z0(), S, P.with_(PR, tau_risk=0.35))
    eta = PR.eta0
    for l in res.log:
        if l.exact and l.bank > 0 and l.support >= PR.n_min and l.finite:
            assert np.isfinite(l.d_cf)
            eta = float(np.clip(PR.beta_d * eta + (1 - PR.beta_d) * l.d_cf / (l.p + PR.eps), PR.eta_min, PR.eta_max))
        else:
            assert np.isnan(l.d_cf)
        assert l.eta == pytest.approx(eta, rel=1e-12)


def test_forced_mask_and_failure_fallbacks():
    S = 8
    mask = [0, 1] * 4
    res = ro.rollout(replay(S), z0(), S, PR, mode="forced", forced=mask)
    assert res.schedule == mask
    # empty support forces exact everywhere (theta_sim above any cosine)
    res2 = ro.rollout(replay(S), z0(), S, P.with_(PR, theta_sim=1.01), mode="forced", forced=[1] * S)
    assert res2.schedule == [0] * S
    # the first step has an empty bank and is exact whatever the mask says
    assert ro.rollout(replay(S), z0(), S, PR, mode="forced", forced=[1] * S).schedule[0] == 0


def test_surrogate_commits_candidate_and_never_inserts():
    S = 8
    trace = []
    res = ro.rollout(replay(S), z0(), S, PR, mode="forced", forced=[0, 1] * 4, trace=trace)
    # step 1 has one record: the committed state is that record's output, i.e. z after step 0
    np.testing.assert_array_equal(trace[1], trace[0])
    assert res.inserts == 4


def test_nonfinite_candidate_falls_back():
    S = 8
    vel = synth.gen_replay_velocities(CFG, S).astype(np.float64)
    vel[0, 0, 0, 0, 0] = np.inf          # the first exact output (the first bank record) is non-finite
    res = ro.rollout(ro.replay_denoiser(vel), z0(), S, PR, mode="forced", forced=[0, 1, 1, 1, 1, 1, 1, 1])
    assert res.schedule[1] == 0 and not res.log[1].finite
