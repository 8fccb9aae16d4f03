"""Property-based pins of the oracle (CPU): hypothesis draws shapes, seeds and
scales (derandomized, so every run draws the same cases) and each property is
one the mathematics fixes, independent of the oracle's own arithmetic:

* attention equals the triple-loop definition, for any head count, query and
  key counts and score scale (large scales test the max subtraction);
* RoPE keeps every vector's norm, and a rotated query-key product depends on
  the two positions only through their difference (Sec. 4.1 backbones);
* the candidate of Eq. (5) is a convex combination of the stored outputs: its
  retrieval and observation weights are non-negative and sum to one, and it
  lies inside the outputs' elementwise hull, for any bank of 1 to 4 records;
* Eq. (6), (9): R_cand = lambda R + w eta p for any inputs, with w in [1, 2];
  Eq. (8): eta stays inside [eta_min, eta_max] for any defect.
"""
import math

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import dit
from oracle import params as P
from oracle import risk as rk
from oracle import surrogate as sg
from tests.test_oracle_dit import brute_attention
from tests.test_oracle_surrogate import make_bank

SETTINGS = settings(max_examples=40, deadline=None, derandomize=True, database=None,
                    suppress_health_check=list(HealthCheck))
PR = P.DEFAULTS


@SETTINGS
@given(heads=st.integers(1, 3), nq=st.integers(1, 9), nk=st.integers(1, 11), hd=st.sampled_from([2, 4, 8]),
       scale=st.sampled_from([0.1, 1.0, 10.0, 60.0]), seed=st.integers(0, 2**32 - 1))
def test_attention_is_the_definition(heads, nq, nk, hd, scale, seed):
    rng = np.random.default_rng(seed)
    q = scale * rng.standard_normal((heads, nq, hd))
    k, v = rng.standard_normal((heads, nk, hd)), rng.standard_normal((heads, nk, hd))
    np.testing.assert_allclose(dit.attention(q, k, v, chunk=4), brute_attention(q, k, v), atol=1e-11, rtol=1e-11)


@SETTINGS
@given(dims=st.sampled_from([(4, 6, 6), (16, 24, 24), (8, 12, 12)]), shift=st.integers(-5, 5),
       seed=st.integers(0, 2**32 - 1))
def test_rope_norm_and_relative_position(dims, shift, seed):
    rng = np.random.default_rng(seed)
    grid = (3, 4, 5)
    hd = sum(dims)
    pos = dit.token_positions(grid).astype(float)
    ang = dit.rope_angles(grid, dims)
    x = rng.standard_normal((1, len(pos), hd))
    np.testing.assert_allclose(np.linalg.norm(dit.apply_rope(x, ang), axis=-1), np.linalg.norm(x, axis=-1),
                               rtol=1e-12)
    # the same rotation computed at every position shifted by `shift` along each axis
    parts = []
    for a, d in enumerate(dims):
        j = np.arange(d // 2)
        parts.append(np.outer(pos[:, a] + shift, dit.ROPE_BASE ** (-2.0 * j / d)))
    ang2 = np.concatenate(parts, 1)
    qv, kv = rng.standard_normal((1, len(pos), hd)), rng.standard_normal((1, len(pos), hd))
    s1 = dit.apply_rope(qv, ang)[0] @ dit.apply_rope(kv, ang)[0].T
    s2 = dit.apply_rope(qv, ang2)[0] @ dit.apply_rope(kv, ang2)[0].T
    np.testing.assert_allclose(s1, s2, atol=1e-10)


@SETTINGS
@given(n=st.integers(1, 4), seed=st.integers(0, 2**32 - 1), dq=st.sampled_from([0.02, 0.05, 0.1]))
def test_candidate_is_a_convex_combination(n, seed, dq):
    rng = np.random.default_rng(seed)
    bank, z, za, h, qa, qam1, q = make_bank(n, rng=rng, dq=dq)
    phi = sg.lift(z, za, h, q, sg.cam_descriptor(None, PR.eps_nu), PR)
    c = sg.candidate(phi, bank, q - dq, qa, qam1, PR)
    outs = np.stack([r.z_out for _, r in bank.records()])
    assert np.all(c.pi >= 0) and np.all(c.kappa >= 0)
    assert math.isclose(float(c.pi.sum()), 1.0, rel_tol=1e-12)
    assert math.isclose(float(c.kappa.sum()), 1.0, rel_tol=1e-12)
    tol = 1e-12 * np.abs(outs).max()
    assert np.all(c.z_hat >= outs.min(0) - tol) and np.all(c.z_hat <= outs.max(0) + tol)


@SETTINGS
@given(R=st.floats(0, 10), eta=st.floats(0.01, 10), p=st.floats(0, 5), q=st.floats(0, 1),
       d_cam=st.floats(0, 3), d_cf=st.floats(0, 50))
def test_accumulation_weight_and_calibration(R, eta, p, q, d_cam, d_cf):
    w = rk.sensitivity_weight(q, PR, d_cam=d_cam)
    assert 1.0 <= w <= 2.0
    d_hat, delta, r_cand = rk.accumulate(R, eta, p, w, PR)
    assert d_hat == eta * p and delta == w * d_hat
    assert math.isclose(r_cand, PR.lam * R + w * eta * p, rel_tol=1e-15, abs_tol=1e-300)
    e2 = rk.calibrate(eta, d_cf, p, PR)
    assert PR.eta_min <= e2 <= PR.eta_max
