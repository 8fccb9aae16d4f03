"""bf16 rollouts that evaluate the real F_theta, against the oracle (GPU).

The risk threshold is swept so that 0 to 60% of the steps take the surrogate
(Eq. (10)); thresholds come from the oracle alone (tests/tau_search.py), at
the centre of the range that reproduces each schedule. The GPU's bf16
F_theta differs from the float64 oracle by bf16 rounding, which moves every
R_cand a little: a threshold is used only when every available step's R_cand
lies at least MIN_MARGIN (relative) away from it, so both sides must take the
same decisions. Bar: schedule bit-exact, final latent within 5e-2 relative
L2."""
import math

import numpy as np
import pytest

import synth
from oracle import params as P
from oracle import rollout as ro
from tests import tau_search as ts
from tests.gpu_util import TOL_BF16_FINAL, rel_l2, small_cfg, torch_cuda

pytestmark = pytest.mark.gpu

MIN_MARGIN = 0.03
# the mid sweep's thresholds (stored oracle rollouts) keep every R_cand at least
# 1.2% away: twenty times the drift measured on the small model
MIN_MARGIN_MID = 0.01


def _rel(a, b):
    return abs(a - b) / max(abs(b), 1e-12)


def compare_bf16_logs(glog, olog):
    """Integer decisions exact; float quantities within the drift bf16 rounding of
    F_theta can cause (returned for the report)."""
    worst = 0.0
    for g, o in zip(glog, olog):
        assert g["exact"] == int(o.exact) and g["bank"] == o.bank and g["support"] == o.support
        assert g["available"] == int(o.available) and g["finite"] == int(o.finite)
        for key in ("d_z", "p", "r_cand", "eta", "R"):
            worst = max(worst, _rel(g[key], getattr(o, key)))
    return worst


def test_small_bf16_rollout_threshold_sweep():
    """The small joint model (all three block kinds, text, camera) in bf16, 10
    steps, thresholds giving 0, 2, 4 and 6 surrogate steps."""
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    cfg = small_cfg("bf16")
    S = 10
    W = synth.gen_weights(cfg)
    inp = synth.gen_inputs(cfg)
    den = ts.memo_denoiser(ro.dit_denoiser(W, cfg, inp), {})
    run = lambda tau: ro.rollout(den, inp["z_T"], S, P.with_(P.DEFAULTS, tau_risk=tau), cam=inp["cam"])
    targets = (0, 2, 4, 6)
    seen = ts.explore(run, budget=60, targets=targets, min_margin=MIN_MARGIN)
    ctx = wdc.Context(cfg)
    ctx.load_weights(W)
    dv = {k: ctx.to_device(inp[k]) for k in ("cond", "text", "cam")}
    for n in targets:
        tau, m = ts.pick(seen, n)
        assert m >= MIN_MARGIN, (n, tau, m)
        ref = run(tau)
        assert sum(ref.schedule) == n
        rctx = wdc.Context(cfg, params=wdc.default_params(tau_risk=tau), allocate_weights=False)
        rctx.bind_weights(ctx.weights)
        z = torch.from_numpy(inp["z_T"]).cuda()
        sched, logs = rctx.rollout(rctx.new_state(), z, S, dv["cond"], dv["text"], dv["cam"], mode=wdc.MODE_RISK)
        err = rel_l2(z.cpu().numpy(), ref.z)
        drift = compare_bf16_logs(logs, ref.log)
        print(f"{n} surrogate steps: tau {tau:.5g} margin {m:.3f} schedule {sched} final rel_l2 {err:.2e} "
              f"log drift {drift:.2e}")
        assert sched == ref.schedule
        assert err <= TOL_BF16_FINAL


def test_mid_bf16_rollout_threshold_sweep():
    """The mid workload (8 blocks, D = 1024, 16 x 64 heads, 2,688 tokens, bf16),
    20 steps, thresholds giving 0, 2, ..., 12 surrogate steps (0-60% skipped).
    The oracle's rollouts (tests/golden/make_tau_sweeps.py) are stored: per
    threshold its schedule, controller log, the final latent at 2,048 fixed
    positions and the final latent's norm."""
    import json
    import os
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "mid_tau_sweep.json")
    gold = json.load(open(path))
    cfg = synth.get_config("mid")
    S = gold["steps"]
    assert gold["workload"] == "mid" and S == 20
    idx = torch.tensor(gold["sample_index"], device="cuda")
    counts = sorted(sum(case["schedule"]) for case in gold["cases"])
    assert counts == list(range(0, 13, 2))
    base = wdc.Context(cfg)
    base.load_weights(synth.gen_weights(cfg))
    inp = synth.gen_inputs(cfg)
    cond = base.to_device(inp["cond"])
    for case in gold["cases"]:
        tau = case["tau"]
        assert case["margin"] >= MIN_MARGIN_MID
        ctx = wdc.Context(cfg, params=wdc.default_params(tau_risk=tau), allocate_weights=False)
        ctx.bind_weights(base.weights)
        z = torch.from_numpy(inp["z_T"]).cuda()
        sched, logs = ctx.rollout(ctx.new_state(), z, S, cond, mode=wdc.MODE_RISK)
        got = z.reshape(-1)[idx].double().cpu().numpy()
        ref = np.asarray(case["final_samples"])
        err = rel_l2(got, ref)
        norm_err = abs(float(z.double().norm()) - case["final_norm"]) / case["final_norm"]
        drift = 0.0
        for g, o in zip(logs, case["log"]):
            assert g["exact"] == int(o["exact"]) and g["bank"] == int(o["bank"]) and g["support"] == int(o["support"])
            assert g["available"] == int(o["available"]) and g["finite"] == int(o["finite"])
            for key in ("d_z", "p", "r_cand", "eta", "R"):
                drift = max(drift, _rel(g[key], o[key]))
        print(f"{sum(sched)} surrogate steps: tau {tau:.5g} margin {case['margin']:.3f} sampled final rel_l2 "
              f"{err:.2e}, norm {norm_err:.2e}, log drift {drift:.2e}")
        assert sched == case["schedule"]
        assert err <= TOL_BF16_FINAL and norm_err <= TOL_BF16_FINAL
        del ctx
