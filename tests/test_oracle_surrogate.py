"""Pins for the oracle surrogate (Eq. (2)-(5)) and risk controller (Eq. (6)-(10)), CPU only."""
import math

import numpy as np
import pytest

from oracle import params as P
from oracle import risk as rk
from oracle import surrogate as sg

RNG = np.random.default_rng(99)
PR = P.DEFAULTS
SHAPE = (16, 3, 5, 7)       # T = 105: chunk sizes are uneven for G = 2, 4, 8


# --------------------------------------------------------------------------- pooling and summaries

def brute_pool(x, G):
    c = x.shape[0]
    flat = x.reshape(c, -1)
    T = flat.shape[1]
    out = []
    for ci in range(c):
        for g in range(G):
            members = [j for j in range(T) if g * T <= j * G < (g + 1) * T]
            out.append(sum(flat[ci, j] for j in members) / math.sqrt(len(members)))
    return np.array(out)


@pytest.mark.parametrize("G", [2, 4, 8, 16])
def test_pool_brute_force(G):
    x = RNG.standard_normal(SHAPE)
    np.testing.assert_allclose(sg.pool(x, G), brute_pool(x, G), atol=1e-12)


def test_pool_nesting_and_energy():
    x = RNG.standard_normal(SHAPE)
    T = 3 * 5 * 7
    j = np.arange(T)
    for G in (2, 4):
        assert np.array_equal((j * G) // T, ((j * 8) // T) // (8 // G))
    # pooling a constant c gives c * sqrt(n): sum of squares of P_G(1) = T per channel
    np.testing.assert_allclose(np.sum(sg.pool(np.ones(SHAPE), 8) ** 2), 16 * T)
    # P_G is linear
    y = RNG.standard_normal(SHAPE)
    np.testing.assert_allclose(sg.pool(2 * x - 3 * y, 4), 2 * sg.pool(x, 4) - 3 * sg.pool(y, 4), atol=1e-12)


def test_nu_and_sim_are_scale_invariant():
    x = RNG.standard_normal(SHAPE)
    np.testing.assert_allclose(sg.nu(7.5 * x, 0.0), sg.nu(x, 0.0), atol=1e-13)
    np.testing.assert_allclose(np.sqrt(np.mean(sg.nu(x, 0.0) ** 2)), 1.0)
    a, b = RNG.standard_normal(256), RNG.standard_normal(256)
    assert sg.sim(3 * a, 0.5 * b) == pytest.approx(sg.sim(a, b), abs=1e-14)
    assert sg.sim(a, a) == pytest.approx(1.0)
    assert sg.sim(a, -a) == pytest.approx(-1.0)
    assert sg.sim(a, np.zeros(256)) == 0.0


def test_summary_layout():
    z, za = RNG.standard_normal(SHAPE), RNG.standard_normal(SHAPE)
    h = RNG.standard_normal(32)
    cam = sg.cam_descriptor(RNG.standard_normal(48), PR.eps_nu)
    phi = sg.lift(z, za, h, 0.7, cam, PR)
    s = sg.summary(phi)
    assert s.shape == (256,)
    np.testing.assert_allclose(s[:128], brute_pool(z / np.sqrt(np.mean(z * z) + 1e-6), 8), atol=1e-12)
    d = z - za
    np.testing.assert_allclose(s[128:192], brute_pool(d / np.sqrt(np.mean(d * d) + 1e-6), 4), atol=1e-12)
    np.testing.assert_array_equal(s[192:224], h)
    np.testing.assert_array_equal(s[224:240], cam)
    np.testing.assert_array_equal(s[240:], 0)
    # no anchor: the displacement block is zero; no camera: zero descriptor
    s0 = sg.summary(sg.lift(z, None, None, 0.7, sg.cam_descriptor(None, 1e-6), PR))
    np.testing.assert_array_equal(s0[128:], 0)


# --------------------------------------------------------------------------- candidate

def make_bank(n, base=None, rng=RNG, q0=1.0, dq=0.05):
    base = rng.standard_normal(SHAPE) if base is None else base
    bank = sg.Bank(4)
    za, h = None, None
    cam = sg.cam_descriptor(None, PR.eps_nu)
    z = base
    for i in range(n):
        zn = z + 0.05 * rng.standard_normal(SHAPE) - 0.02 * base
        q, qn = q0 - i * dq, q0 - (i + 1) * dq
        pin, pout = sg.lift(z, za, h, q, cam, PR), sg.lift(zn, za, h, qn, cam, PR)
        bank.insert(sg.Record(pin, pout, sg.summary(pin), sg.summary(pout), q, qn, zn))
        h = sg.history_summary(z, zn, PR)
        za, qa, qam1 = z, q, qn
        z = zn
    return bank, z, za, h, qa, qam1, q0 - n * dq


def test_single_record_returns_its_output_bitwise():
    bank, z, za, h, qa, qam1, q = make_bank(1)
    phi = sg.lift(z, za, h, q, np.zeros(16), PR)
    c = sg.candidate(phi, bank, q - 0.05, qa, qam1, PR)
    assert c.kappa.tolist() == [1.0]
    np.testing.assert_array_equal(c.z_hat, bank.slots[0].z_out)


def test_weights_convex_and_candidate_in_hull():
    bank, z, za, h, qa, qam1, q = make_bank(4)
    phi = sg.lift(z, za, h, q, np.zeros(16), PR)
    c = sg.candidate(phi, bank, q - 0.05, qa, qam1, PR)
    assert np.all(c.pi >= 0) and np.all(c.kappa >= 0)
    assert c.pi.sum() == pytest.approx(1.0) and c.kappa.sum() == pytest.approx(1.0)
    outs = np.stack([r.z_out for _, r in bank.records()])
    assert np.all(c.z_hat >= outs.min(0) - 1e-12) and np.all(c.z_hat <= outs.max(0) + 1e-12)
    np.testing.assert_allclose(c.z_hat, np.tensordot(c.kappa, outs, 1), atol=1e-13)


def test_retrieval_weights_closed_form():
    bank, z, za, h, qa, qam1, q = make_bank(3)
    phi = sg.lift(z, za, h, q, np.zeros(16), PR)
    c = sg.candidate(phi, bank, q - 0.05, qa, qam1, PR)
    s = sg.summary(phi)
    ell = [sg.sim(s, r.s_in) - PR.gamma_q * (q - r.q_in) ** 2 for _, r in bank.records()]
    e = np.exp(np.array(ell) / PR.tau_in)
    np.testing.assert_allclose(c.pi, e / e.sum(), rtol=1e-12)
    kap = np.exp(np.array([sg.sim(c.s_hat, r.s_out) for _, r in bank.records()]) / PR.tau_obs)
    np.testing.assert_allclose(c.kappa, kap / kap.sum(), rtol=1e-12)


def test_alpha_on_uniform_grid():
    S = 20
    a = sg.scheduler_scale(1 - 5 / S, 1 - 6 / S, 1 - 3 / S, 1 - 4 / S, PR)
    assert a == pytest.approx((1 / S) / (1 / S + PR.eps), rel=1e-12)
    assert sg.scheduler_scale(0.5, 0.3, 0.6, 0.55, PR) == PR.alpha_max      # 0.2/0.05 = 4 -> clipped
    assert sg.scheduler_scale(0.5, 0.49, 0.6, 0.5, PR) == PR.alpha_min      # 0.01/0.1 -> clipped


def test_summary_space_evolution_equals_full_size():
    """s is linear, so s(phi_hat) = s(phi_t) + alpha * sum pi_i (s_out_i - s_in_i)."""
    bank, z, za, h, qa, qam1, q = make_bank(4)
    phi = sg.lift(z, za, h, q, np.zeros(16), PR)
    c = sg.candidate(phi, bank, q - 0.05, qa, qam1, PR)
    lin = sg.summary(phi) + c.alpha * sum(c.pi[j] * (r.s_out - r.s_in) for j, (_, r) in enumerate(bank.records()))
    np.testing.assert_allclose(c.s_hat, lin, atol=1e-12)


def test_support_thresholds():
    bank, z, za, h, qa, qam1, q = make_bank(3)
    phi = sg.lift(z, za, h, q, np.zeros(16), PR)
    assert sg.candidate(phi, bank, q - 0.05, qa, qam1, P.with_(PR, theta_sim=1.01)).support == []
    # phase window: only records whose input phase is within theta_q
    c = sg.candidate(phi, bank, q - 0.05, qa, qam1, P.with_(PR, theta_q=0.11, theta_sim=-1.0))
    qs = [r.q_in for _, r in bank.records()]
    assert c.support == [i for i, qi in enumerate(qs) if abs(q - qi) <= 0.11]
    # unsupported records get no retrieval weight, and the lifted state does not move
    c0 = sg.candidate(phi, bank, q - 0.05, qa, qam1, P.with_(PR, theta_sim=1.01))
    np.testing.assert_array_equal(c0.pi, 0)
    np.testing.assert_allclose(c0.s_hat, sg.summary(phi), atol=0)


def test_nonfinite_bank_output_marks_candidate():
    bank, z, za, h, qa, qam1, q = make_bank(2)
    bank.slots[1].z_out = bank.slots[1].z_out.copy()
    bank.slots[1].z_out[0, 0, 0, 0] = np.nan
    phi = sg.lift(z, za, h, q, np.zeros(16), PR)
    assert not sg.candidate(phi, bank, q - 0.05, qa, qam1, PR).finite


def test_fifo_slots():
    b = sg.Bank(4)
    slots = [b.insert(i) for i in range(10)]
    assert slots == [0, 1, 2, 3, 0, 1, 2, 3, 0, 1]
    assert b.slots == [8, 9, 6, 7]


# --------------------------------------------------------------------------- risk

def test_weight_range_and_cap():
    for q in np.linspace(0, 1, 11):
        w = rk.sensitivity_weight(q, PR)
        assert 1.0 <= w <= 2.0
        assert w == pytest.approx(1 + 0.5 * q)
    assert rk.sensitivity_weight(1.0, PR, d_cam=5.0, d_depth=5.0) == 2.0


def test_calibration_closed_form_and_clamp():
    r, eta = 0.7, 3.0
    prox = 0.25
    for n in range(1, 12):
        eta = rk.calibrate(eta, r * (prox + PR.eps), prox, PR)
        assert eta == pytest.approx(r + PR.beta_d ** n * (3.0 - r), rel=1e-12)
    assert rk.calibrate(1.0, 1e6, 1e-3, PR) == PR.eta_max
    assert rk.calibrate(PR.eta_min, 0.0, 1.0, PR) == PR.eta_min


def test_accumulation_closed_form():
    R = 0.0
    d = 0.03
    for n in range(1, 15):
        _, delta, R = rk.accumulate(R, 1.0, d, 1.0, PR)
        assert R == pytest.approx(d * (1 - PR.lam ** n) / (1 - PR.lam), rel=1e-12)


def test_counterfactual_defect():
    z = RNG.standard_normal(SHAPE)
    assert rk.counterfactual_defect(z, z, 1e-8) == 0.0
    zc = z + 0.1 * RNG.standard_normal(SHAPE)
    d = rk.counterfactual_defect(z, zc, 0.0)
    assert rk.counterfactual_defect(4 * z, 4 * zc, 0.0) == pytest.approx(d, rel=1e-12)
    assert d == pytest.approx(np.abs(z - zc).sum() / np.abs(z).sum(), rel=1e-12)


def test_local_proxy_terms():
    z, za = RNG.standard_normal(SHAPE), RNG.standard_normal(SHAPE)
    pr = rk.local_proxy(z, za, 3, 0.4, 0.55, PR)
    assert pr.d_z == pytest.approx(np.abs(z - za).sum() / (np.abs(za).sum() + PR.eps))
    assert pr.d_age == pytest.approx(4 / 7)
    assert pr.d_phase == pytest.approx(0.15)
    assert pr.p == pytest.approx(pr.d_z + 0.05 * 4 / 7 + 0.5 * 0.15)
    assert rk.local_proxy(z, None, 0, 1.0, 0.0, PR).d_z == 0.0


def test_decision_rule():
    assert rk.decide(True, 0.5, 0.5)          # inclusive threshold
    assert not rk.decide(True, 0.5000001, 0.5)
    assert not rk.decide(False, 0.0, 0.5)
    assert not rk.available(0, 0, 1, True, 3, 10, PR)            # empty bank
    assert not rk.available(2, 7, 1, True, 3, 10, PR)            # anchor too old
    assert rk.available(2, 6, 1, True, 3, 10, PR)
    assert not rk.available(2, 0, 0, True, 3, 10, PR)            # no support
    assert not rk.available(2, 0, 1, False, 3, 10, PR)           # non-finite candidate
    assert not rk.available(2, 0, 1, True, 0, 10, PR)            # initialisation phase
    assert not rk.available(2, 0, 1, True, 9, 10, P.with_(PR, k_ref=1))   # refinement phase
