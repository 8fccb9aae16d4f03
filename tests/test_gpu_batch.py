"""GPU parity of batched rollouts (several latents with per-sample schedules,
F_theta evaluated once per step over the exact subset): the batched forward
against per-sample forwards and the oracle, and batched rollouts against the
oracle's independent per-sample rollouts."""
from dataclasses import replace

import numpy as np
import pytest

import synth
from oracle import dit
from oracle import params as P
from oracle import rollout as ro
from tests.gpu_util import TOL_BF16_FINAL, TOL_F32, rel_l2, small_cfg, torch_cuda, wdc_params

pytestmark = pytest.mark.gpu


def seeded(cfg, b):
    return replace(cfg, seed=cfg.seed + 17 * b + 1)


def batch_context(cfg, B, params=None, weights=True):
    torch_cuda()
    import paper_2608_01845_amd as wdc
    ctx = wdc.Context(cfg, params=params, allocate_weights=weights, max_batch=B)
    if weights:
        ctx.load_weights(synth.gen_weights(cfg))
    return ctx


def inputs(ctx, cfg, B):
    import torch
    host, dev = [], []
    for b in range(B):
        inp = synth.gen_inputs(seeded(cfg, b))
        host.append(inp)
        dev.append({"z_T": ctx.to_device(inp["z_T"], dtype=torch.float32),
                    **{k: ctx.to_device(inp[k]) for k in ("cond", "text", "cam") if k in inp}})
    return host, dev


def lists(dev, key):
    vals = [d.get(key) for d in dev]
    return None if all(v is None for v in vals) else vals


@pytest.mark.parametrize("cfg_name,B", [("tiny", 3), ("unit64", 3), ("unit128", 4)])
def test_forward_batch_equals_single_forwards(cfg_name, B):
    cfg = {"tiny": lambda: synth.get_config("tiny"), "unit64": lambda: small_cfg(head_dim=64),
           "unit128": lambda: small_cfg(head_dim=128)}[cfg_name]()
    ctx = batch_context(cfg, B)
    host, dev = inputs(ctx, cfg, B)
    zs = [d["z_T"] for d in dev]
    t = 0.625
    outs = ctx.forward_batch(zs, t, lists(dev, "cond"), lists(dev, "text"), lists(dev, "cam"))
    for b in range(B):
        single = ctx.forward(zs[b], t, dev[b].get("cond"), dev[b].get("text"), dev[b].get("cam"))
        err = rel_l2(outs[b].cpu().numpy(), single.cpu().numpy())
        print(cfg_name, "sample", b, "batched vs single rel_l2", err)
        assert err <= 1e-5
    # one sample against the oracle
    W = synth.gen_weights(cfg)
    ref = dit.dit_forward(W, cfg, host[B - 1]["z_T"], t, host[B - 1].get("cond"), host[B - 1].get("text"),
                          host[B - 1].get("cam"))
    err = rel_l2(outs[B - 1].cpu().numpy(), ref)
    print(cfg_name, "batched vs oracle", err)
    assert err <= (TOL_F32 if cfg.dtype == "f32" else TOL_BF16_FINAL)


def test_rollout_batch_per_sample_masks_tiny_dit():
    """Different forced masks per sample: the exact subset changes size every step."""
    import paper_2608_01845_amd as wdc
    cfg = synth.get_config("tiny")
    S, B = 8, 3
    masks = [[0, 1] * 4, [0, 0, 1, 1, 0, 1, 1, 1], [0, 1, 1, 0, 1, 0, 0, 1]]
    ctx = batch_context(cfg, B)
    host, dev = inputs(ctx, cfg, B)
    zs = [d["z_T"].clone() for d in dev]
    states = [ctx.new_state() for _ in range(B)]
    scheds, logs = ctx.rollout_batch(states, zs, S, lists(dev, "cond"), mode=wdc.MODE_FORCED, forced=masks)
    W = synth.gen_weights(cfg)
    for b in range(B):
        ref = ro.rollout(ro.dit_denoiser(W, cfg, host[b]), host[b]["z_T"], S, P.DEFAULTS, mode="forced",
                         forced=masks[b])
        assert scheds[b] == ref.schedule == masks[b]
        for g, o in zip(logs[b], ref.log):
            assert g["exact"] == int(o.exact) and g["bank"] == o.bank and g["support"] == o.support
            for key in ("d_z", "p", "r_cand", "eta", "R"):
                assert abs(g[key] - getattr(o, key)) <= 1e-4 * max(1.0, abs(getattr(o, key))), (b, key)
        err = rel_l2(zs[b].cpu().numpy(), ref.z)
        print("sample", b, "final rel_l2", err)
        assert err <= TOL_F32


def test_rollout_batch_risk_mode_matches_single_rollouts():
    """Risk-controlled decisions per sample: batched = each sample alone (same τ)."""
    import paper_2608_01845_amd as wdc
    cfg = synth.get_config("tiny")
    S, B = 12, 3
    W = synth.gen_weights(cfg)
    host = [synth.gen_inputs(seeded(cfg, b)) for b in range(B)]
    dens = [ro.dit_denoiser(W, cfg, h) for h in host]
    # a threshold whose oracle margins are clear for every sample
    rng = np.random.default_rng(0)
    tau = None
    for _ in range(100):
        cand = float(rng.uniform(0.1, 1.0))
        refs = [ro.rollout(d, h["z_T"], S, P.with_(P.DEFAULTS, tau_risk=cand)) for d, h in zip(dens, host)]
        if all(min((l.margin for l in r.log if l.available), default=np.inf) >= 1e-3 for r in refs) and \
                any(sum(r.schedule) for r in refs):
            tau = cand
            break
    assert tau is not None
    ctx = batch_context(cfg, B, params=wdc.default_params(tau_risk=tau))
    _, dev = inputs(ctx, cfg, B)
    zs = [d["z_T"].clone() for d in dev]
    scheds, _ = ctx.rollout_batch([ctx.new_state() for _ in range(B)], zs, S, lists(dev, "cond"),
                                  mode=wdc.MODE_RISK)
    print("tau", tau, "schedules", scheds)
    for b in range(B):
        assert scheds[b] == refs[b].schedule
        assert rel_l2(zs[b].cpu().numpy(), refs[b].z) <= TOL_F32
        z1 = dev[b]["z_T"].clone()
        s1, _ = ctx.rollout(ctx.new_state(), z1, S, dev[b]["cond"], mode=wdc.MODE_RISK)
        assert s1 == scheds[b]
        assert rel_l2(zs[b].cpu().numpy(), z1.cpu().numpy()) <= 1e-5


def test_rollout_batch_replay_mid_latent():
    """Recorded velocities per sample on the mid latent, periodic placement."""
    import torch
    import paper_2608_01845_amd as wdc
    cfg = synth.get_config("mid")
    S, B = 20, 4
    p = P.with_(P.DEFAULTS, period=4, surrogate="secant")
    ctx = batch_context(cfg, B, params=wdc_params(p), weights=False)
    zs, vels, refs = [], [], []
    for b in range(B):
        c = seeded(cfg, b)
        z0 = synth.gen_inputs(c)["z_T"]
        vel = synth.gen_replay_velocities(c, S)
        refs.append(ro.rollout(ro.replay_denoiser(vel), z0, S, p, mode="periodic"))
        zs.append(torch.from_numpy(z0).cuda())
        vels.append(torch.from_numpy(vel).cuda())
    scheds, _ = ctx.rollout_batch([ctx.new_state() for _ in range(B)], zs, S, mode=wdc.MODE_PERIODIC,
                                  replay_vs=vels)
    for b in range(B):
        assert scheds[b] == refs[b].schedule
        assert rel_l2(zs[b].cpu().numpy(), refs[b].z) <= TOL_F32


def test_batch_larger_than_max_batch_is_rejected():
    import paper_2608_01845_amd as wdc
    cfg = synth.get_config("tiny")
    ctx = batch_context(cfg, 2)
    _, dev = inputs(ctx, cfg, 3)
    with pytest.raises(wdc.WdcError):
        ctx.forward_batch([d["z_T"] for d in dev], 0.5, lists(dev, "cond"))
