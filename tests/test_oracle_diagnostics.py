"""Pins for the synthetic risk diagnostics (Observation 1, Sec. 3; calibration
diagnostics, Sec. 4.3), CPU only: the oracle's injection sweep against what
the Euler structure fixes, and both sides' statistics against scipy and brute
force."""
import numpy as np
import pytest
from scipy import stats

import synth
from oracle import diagnostics as od
from oracle import params as P
from oracle import rollout as ro
from paper_2608_01845_amd import diagnostics as gd

CFG = synth.get_config("tiny")


def z0():
    return synth.gen_inputs(CFG)["z_T"]


@pytest.mark.parametrize("mod", [od, gd])
def test_correlations_match_scipy(mod):
    rng = np.random.default_rng(0)
    x = rng.standard_normal(40)
    y = 0.6 * x + rng.standard_normal(40)
    y[:5] = y[5]                     # ties
    assert mod.pearson(x, y) == pytest.approx(stats.pearsonr(x, y)[0], rel=1e-12)
    assert mod.spearman(x, y) == pytest.approx(stats.spearmanr(x, y)[0], rel=1e-12)


@pytest.mark.parametrize("mod,fn", [(od, "false_safe_rates"), (gd, "false_safe")])
def test_false_safe_brute_force(mod, fn):
    crit = [0.1, 0.2, 0.3, 0.4, 0.5, 0.6]
    down = [0.9, 0.1, 0.8, 0.2, 0.7, 0.3]
    phase = [0.05, 0.2, 0.5, 0.6, 0.9, 0.95]
    r = getattr(mod, fn)(crit, down, phase)
    # median crit 0.35: safe = first three; median down 0.5: bad = 0.9, 0.8, 0.7
    assert r["all"] == pytest.approx(2 / 3)
    assert r["phase_bin0"] == pytest.approx(1 / 2)      # phases 0.05 (bad), 0.2 (good)
    assert r["phase_bin1"] == pytest.approx(1.0)        # phase 0.5 (bad)
    assert np.isnan(r["phase_bin2"])                    # no safe step late


def test_replay_downstream_equals_carried_local_defect():
    """With F_theta independent of z, the injected error is carried unchanged to
    the end: mean|z'_0 - z_0| = mean|z_hat - z_{t+1}| for every injected t."""
    S = 12
    vel = synth.gen_replay_velocities(CFG, S)
    den = ro.replay_denoiser(vel)
    sw = od.injection_sweep(den, z0(), S, P.DEFAULTS)
    assert sw["step"] == list(range(1, S))
    trace = []
    ref = ro.rollout(den, z0(), S, P.DEFAULTS, mode="all_exact", trace=trace)
    eps = P.DEFAULTS.eps
    for t, dl, dd in zip(sw["step"], sw["d_local"], sw["down"]):
        carried = dl * (np.mean(np.abs(trace[t])) + eps)
        assert dd * (np.mean(np.abs(ref.z)) + eps) == pytest.approx(carried, rel=1e-10)
    # local defects equal the all-exact rollout's counterfactual defects
    np.testing.assert_allclose(sw["d_local"], [ref.log[t].d_cf for t in sw["step"]], rtol=1e-12)
    assert len(sw["anchor_d_cf"]) == sum(np.isfinite(l.d_cf) for l in ref.log) == S - 1


def test_secant_on_constant_velocity_has_no_defect_anywhere():
    S = 8
    v = synth.gen_replay_velocities(CFG, 1)[0]
    sw = od.injection_sweep(ro.replay_denoiser(np.stack([v] * S)), z0(), S,
                            P.with_(P.DEFAULTS, surrogate="secant"))
    assert len(sw["step"]) == S - 1
    assert max(sw["d_local"]) < 1e-13 and max(sw["down"]) < 1e-13


def test_weighted_criterion_is_local_times_weight():
    S = 10
    vel = synth.gen_replay_velocities(CFG, S)
    sw = od.injection_sweep(ro.replay_denoiser(vel), z0(), S, P.DEFAULTS)
    q = np.array(sw["phase"])
    w = np.minimum(2.0, 1.0 + P.DEFAULTS.a_phase * q)
    np.testing.assert_allclose(sw["delta"], w * np.array(sw["d_hat"]), rtol=1e-14)
