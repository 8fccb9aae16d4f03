"""GPU parity of the synthetic risk diagnostics and the matched-budget
factorization (Observation 1, Sec. 3; Sec. 5.4) on the tiny float32 DiT: the
injection sweep's per-step quantities and the factorization's final-latent
errors against the oracle."""
import numpy as np
import pytest

import synth
from oracle import diagnostics as od
from oracle import params as P
from oracle import rollout as ro
from tests.gpu_util import context, dev_inputs, torch_cuda, wdc_params

pytestmark = pytest.mark.gpu


def setup(cfg_name="tiny", params=P.DEFAULTS):
    torch_cuda()
    from paper_2608_01845_amd import diagnostics as gd
    cfg = synth.get_config(cfg_name)
    W = synth.gen_weights(cfg)
    inp = synth.gen_inputs(cfg)
    ctx = context(cfg, params=wdc_params(params))
    _, dv = dev_inputs(ctx, cfg)
    gin = gd.Inputs(dv["z_T"], dv["cond"], dv["text"], dv["cam"])
    return gd, cfg, W, inp, ctx, gin


def test_injection_sweep_matches_oracle():
    gd, cfg, W, inp, ctx, gin = setup()
    S = 8
    g = gd.injection_sweep(ctx, gin, S)
    o = od.injection_sweep(ro.dit_denoiser(W, cfg, inp), inp["z_T"], S, P.DEFAULTS)
    print("steps", g.step, "down", np.round(g.down, 5), "local", np.round(g.d_local, 5))
    assert g.step == o["step"]
    for key in ("phase", "d_local", "d_hat", "delta", "down", "anchor_d_hat", "anchor_d_cf"):
        np.testing.assert_allclose(getattr(g, key), o[key], rtol=1e-3, atol=1e-6, err_msg=key)
    s = g.summary()
    assert s["pearson_dhat_dcf"] == pytest.approx(od.pearson(o["anchor_d_hat"], o["anchor_d_cf"]), abs=1e-3)
    assert s["spearman_down_weighted"] == pytest.approx(od.spearman(o["delta"], o["down"]), abs=1e-6)


def test_factorization_periodic_matches_oracle_and_budget():
    gd, cfg, W, inp, ctx, gin = setup()
    S, period = 8, 2
    res = gd.factorization(ctx, gin, S, period)
    print(res)
    den = ro.dit_denoiser(W, cfg, inp)
    ref = ro.rollout(den, inp["z_T"], S, P.DEFAULTS, mode="all_exact")
    for cons in ("lifted", "secant"):
        o = ro.rollout(den, inp["z_T"], S, P.with_(P.DEFAULTS, surrogate=cons, period=period), mode="periodic")
        r = res[f"periodic+{cons}"]
        assert r["exact_calls"] == S - sum(o.schedule) == 4
        oerr = float(np.mean(np.abs(o.z - ref.z)) / (np.mean(np.abs(ref.z)) + 1e-8))
        assert r["l1_rel"] == pytest.approx(oerr, rel=1e-3, abs=1e-6)
        rr = res[f"risk+{cons}"]
        assert abs(rr["exact_calls"] - 4) <= 1
        # the same threshold in the oracle, compared when no decision sits near it
        o2 = ro.rollout(den, inp["z_T"], S, P.with_(P.DEFAULTS, surrogate=cons, tau_risk=rr["tau_risk"]))
        if min((l.margin for l in o2.log if l.available), default=np.inf) >= 1e-3:
            assert S - sum(o2.schedule) == rr["exact_calls"]
            oerr2 = float(np.mean(np.abs(o2.z - ref.z)) / (np.mean(np.abs(ref.z)) + 1e-8))
            assert rr["l1_rel"] == pytest.approx(oerr2, rel=1e-3, abs=1e-6)
