"""Block, forward and rollout parity of the HIP path against the oracle (GPU)."""
import numpy as np
import pytest

import synth
from oracle import dit
from oracle import params as P
from oracle import rollout as ro
from tests.gpu_util import (TOL_BF16_BLOCK, TOL_BF16_FINAL, TOL_F32, context, dev_inputs, pick_tau, rel_l2,
                            small_cfg, torch_cuda)

pytestmark = pytest.mark.gpu


def run_block(ctx, cfg, block, x, c):
    torch = torch_cuda()
    xd = torch.from_numpy(np.ascontiguousarray(x, np.float32)).cuda()
    cd = torch.from_numpy(np.ascontiguousarray(c, np.float32)).cuda()
    ctx.block_forward(block, xd, cd)
    return xd.cpu().numpy()


@pytest.mark.parametrize("dtype,head_dim", [("f32", 64), ("bf16", 64), ("bf16", 128), ("f32", 128)])
def test_every_block_kind_matches_oracle(dtype, head_dim):
    cfg = small_cfg(dtype, head_dim=head_dim)
    ctx = context(cfg)
    W = synth.gen_weights(cfg)
    x = synth.gen_block_input(cfg)
    c = synth.gen_cemb(cfg)
    for b in range(cfg.n_blocks):
        got = run_block(ctx, cfg, b, x, c)
        ref = dit.block_forward(W, cfg, b, x, c)
        err, derr = rel_l2(got, ref), rel_l2(got - x, ref - x)
        print(f"{dtype} hd={head_dim} block {b} ({dit.block_kind(cfg, b)}): rel_l2 {err:.2e}, update rel_l2 {derr:.2e}")
        if dtype == "f32":
            assert err <= TOL_F32 and derr <= 1e-3
        else:
            assert err <= TOL_BF16_BLOCK and derr <= 5e-2


def test_tiny_forward_matches_oracle():
    torch = torch_cuda()
    cfg = synth.get_config("tiny")
    ctx = context(cfg)
    W = synth.gen_weights(cfg)
    inp, dv = dev_inputs(ctx, cfg)
    for t in (1.0, 0.375):
        got = ctx.forward(dv["z_T"], t, dv["cond"]).cpu().numpy()
        ref = dit.dit_forward(W, cfg, inp["z_T"], t, inp["cond"])
        assert rel_l2(got, ref) <= TOL_F32


def test_small_joint_forward_matches_oracle():
    cfg = small_cfg("bf16")
    ctx = context(cfg)
    W = synth.gen_weights(cfg)
    inp, dv = dev_inputs(ctx, cfg)
    got = ctx.forward(dv["z_T"], 0.7, dv["cond"], dv["text"], dv["cam"]).cpu().numpy()
    ref = dit.dit_forward(W, cfg, inp["z_T"], 0.7, inp["cond"], inp["text"], inp["cam"])
    err = rel_l2(got, ref)
    print("small joint forward rel_l2", err)
    assert err <= TOL_BF16_FINAL


def test_mid_block_matches_oracle():
    cfg = synth.get_config("mid")
    ctx = context(cfg)
    W = synth.gen_weights(cfg, names=["seq.3"])
    x = synth.gen_block_input(cfg)
    c = synth.gen_cemb(cfg)
    got = run_block(ctx, cfg, 3, x, c)
    ref = dit.block_forward(W, cfg, 3, x, c)
    err, derr = rel_l2(got, ref), rel_l2(got - x, ref - x)
    print(f"mid block 3: rel_l2 {err:.2e}, update {derr:.2e}")
    assert err <= TOL_BF16_BLOCK


def compare_logs(glog, olog, exact_tol):
    assert glog["exact"] == int(olog.exact)
    assert glog["bank"] == olog.bank
    assert glog["support"] == olog.support
    assert glog["available"] == int(olog.available)
    for key in ("d_z", "p", "r_cand", "eta", "R"):
        a, b = glog[key], getattr(olog, key)
        assert abs(a - b) <= exact_tol * max(1.0, abs(b)), (key, a, b)
    if olog.bank:
        np.testing.assert_allclose(glog["kappa"], olog.kappa, atol=exact_tol * 10)
        np.testing.assert_allclose(glog["sims_in"], olog.sims_in, atol=exact_tol)


def test_tiny_forced_rollout_matches_oracle():
    """Anchors at even steps, surrogate + risk at odd steps (8 Euler steps)."""
    torch = torch_cuda()
    cfg = synth.get_config("tiny")
    ctx = context(cfg)
    W = synth.gen_weights(cfg)
    inp, dv = dev_inputs(ctx, cfg)
    mask = [0, 1] * 4
    ref = ro.rollout(ro.dit_denoiser(W, cfg, inp), inp["z_T"], 8, P.DEFAULTS, mode="forced", forced=mask)
    st = ctx.new_state()
    z = dv["z_T"].clone()
    import paper_2608_01845_amd as wdc
    sched, logs = ctx.rollout(st, z, 8, dv["cond"], mode=wdc.MODE_FORCED, forced=mask)
    assert sched == ref.schedule == mask
    for g, o in zip(logs, ref.log):
        compare_logs(g, o, 1e-4)
    assert rel_l2(z.cpu().numpy(), ref.z) <= TOL_F32


def test_tiny_risk_rollout_matches_oracle():
    torch = torch_cuda()
    cfg = synth.get_config("tiny")
    W = synth.gen_weights(cfg)
    inp = synth.gen_inputs(cfg)
    den = ro.dit_denoiser(W, cfg, inp)
    tau, ref = pick_tau(lambda tau: ro.rollout(den, inp["z_T"], 8, P.with_(P.DEFAULTS, tau_risk=tau)),
                        lo=0.05, hi=1.0, target_surrogates=3)
    import paper_2608_01845_amd as wdc
    ctx = context(cfg, params=wdc.default_params(tau_risk=tau))
    _, dv = dev_inputs(ctx, cfg)
    st = ctx.new_state()
    z = dv["z_T"].clone()
    sched, logs = ctx.rollout(st, z, 8, dv["cond"], mode=wdc.MODE_RISK)
    print("tau", tau, "schedule", sched, "oracle", ref.schedule)
    assert sched == ref.schedule
    for g, o in zip(logs, ref.log):
        compare_logs(g, o, 1e-4)
    assert rel_l2(z.cpu().numpy(), ref.z) <= TOL_F32


@pytest.mark.parametrize("name,steps", [("tiny", 50), ("mid", 20)])
def test_replay_rollout_schedule_and_latent(name, steps):
    """Recorded velocities in place of F_theta: the control path at the workload's latent size."""
    torch = torch_cuda()
    cfg = synth.get_config(name)
    vel = synth.gen_replay_velocities(cfg, steps)
    z0 = synth.gen_inputs(cfg)["z_T"]
    den = ro.replay_denoiser(vel)
    tau, ref = pick_tau(lambda tau: ro.rollout(den, z0, steps, P.with_(P.DEFAULTS, tau_risk=tau)), lo=0.05, hi=1.5,
                        target_surrogates=steps // 2)
    import paper_2608_01845_amd as wdc
    ctx = context(cfg, weights=False, params=wdc.default_params(tau_risk=tau))
    st = ctx.new_state()
    z = torch.from_numpy(z0).cuda()
    vd = torch.from_numpy(vel).cuda()
    sched, logs = ctx.rollout(st, z, steps, mode=wdc.MODE_RISK, replay_v=vd)
    print(name, "tau", tau, "surrogates", sum(sched), "of", steps)
    assert sched == ref.schedule
    for g, o in zip(logs, ref.log):
        compare_logs(g, o, 1e-4)
    assert rel_l2(z.cpu().numpy(), ref.z) <= TOL_F32


def test_open_threshold_replay_schedule_is_paper_ratio():
    """tau = inf at 50 steps: 7 exact calls (the paper's 14% exact-call ratio)."""
    torch = torch_cuda()
    cfg = synth.get_config("tiny")
    vel = synth.gen_replay_velocities(cfg, 50)
    import paper_2608_01845_amd as wdc
    ctx = context(cfg, weights=False, params=wdc.default_params(tau_risk=float("inf")))
    z = torch.from_numpy(synth.gen_inputs(cfg)["z_T"]).cuda()
    sched, _ = ctx.rollout(ctx.new_state(), z, 50, mode=wdc.MODE_RISK, replay_v=torch.from_numpy(vel).cuda())
    assert [k for k, s in enumerate(sched) if s == 0] == [0, 8, 16, 24, 32, 40, 48]


def test_all_exact_rollout_equals_plain_euler_bitwise():
    """Candidates are still built every step but must not touch the committed state."""
    torch = torch_cuda()
    cfg = synth.get_config("tiny")
    vel = synth.gen_replay_velocities(cfg, 8)
    import paper_2608_01845_amd as wdc
    ctx = context(cfg, weights=False)
    z0 = torch.from_numpy(synth.gen_inputs(cfg)["z_T"]).cuda()
    vd = torch.from_numpy(vel).cuda()
    z = z0.clone()
    sched, logs = ctx.rollout(ctx.new_state(), z, 8, mode=wdc.MODE_ALL_EXACT, replay_v=vd)
    assert sched == [0] * 8
    ref = z0.clone()
    for k in range(8):
        ref = ctx.scheduler_step(ref, vd[k], (8 - k) / 8, (8 - k - 1) / 8)
    assert torch.equal(z, ref)


def test_nonfinite_bank_latent_forces_exact():
    """A NaN planted (from the host) in a stored exact output makes the candidate
    non-finite, so the step is unavailable and falls back to exact."""
    torch = torch_cuda()
    cfg = synth.get_config("tiny")
    import paper_2608_01845_amd as wdc
    ctx = context(cfg, weights=False)
    st = ctx.new_state()
    vel = torch.from_numpy(synth.gen_replay_velocities(cfg, 8)).cuda()
    z = torch.from_numpy(synth.gen_inputs(cfg)["z_T"]).cuda()
    zhat = torch.empty_like(z)
    ctx.surrogate_step(st, z, 0, 8, zhat)
    assert ctx.risk_update(st, wdc.PRE_DECISION, 0, 8)["exact"] == 1      # empty bank
    zn = ctx.scheduler_step(z, vel[0], 1.0, 0.875)
    ctx.risk_update(st, wdc.POST_EXACT, 0, 8, z, zn)
    ptr, ins = st.bank_slot(0)
    assert ins == 1
    host = torch.empty(cfg.numel, dtype=torch.float32, device="cuda")
    _copy(host.data_ptr(), ptr, cfg.numel)
    assert torch.equal(host, zn.reshape(-1))                              # the slot holds z_1 exactly
    host[17] = float("nan")
    _copy(ptr, host.data_ptr(), cfg.numel)
    log = ctx.surrogate_step(st, zn, 1, 8, zhat)
    assert log["bank"] == 1 and log["finite"] == 0
    log = ctx.risk_update(st, wdc.PRE_DECISION, 1, 8)
    assert log["available"] == 0 and log["exact"] == 1


def _copy(dst_ptr, src_ptr, n):
    import ctypes as C
    torch = torch_cuda()
    torch.cuda.synchronize()
    hip = C.CDLL("libamdhip64.so")
    assert hip.hipMemcpy(C.c_void_p(dst_ptr), C.c_void_p(src_ptr), C.c_size_t(4 * n), 3) == 0   # device to device


@pytest.mark.parametrize("steps", [1, 2, 3])
def test_short_rollouts_match_oracle(steps):
    """The degenerate lengths: S = 1 (one exact step, nothing to reuse), S = 2
    (the only step after the first is the last one) and S = 3, in every mode
    (risk with an open threshold, forced surrogates everywhere, all exact,
    periodic with period 2): schedule, logs and latent against the oracle."""
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    cfg = synth.get_config("tiny")
    W = synth.gen_weights(cfg)
    inp = synth.gen_inputs(cfg)
    den = ro.dit_denoiser(W, cfg, inp)
    cases = [("risk", wdc.MODE_RISK, dict(tau_risk=1e9), None),
             ("forced", wdc.MODE_FORCED, {}, [1] * steps),
             ("all_exact", wdc.MODE_ALL_EXACT, {}, None),
             ("periodic", wdc.MODE_PERIODIC, dict(period=2), None)]
    for name, mode, over, forced in cases:
        ref = ro.rollout(den, inp["z_T"], steps, P.with_(P.DEFAULTS, **over), mode=name, forced=forced)
        ctx = context(cfg, params=wdc.default_params(**over))
        _, dv = dev_inputs(ctx, cfg)
        z = dv["z_T"].clone()
        sched, logs = ctx.rollout(ctx.new_state(), z, steps, dv["cond"], mode=mode, forced=forced)
        print(f"S={steps} {name}: schedule {sched} oracle {ref.schedule}")
        assert sched == ref.schedule and sched[0] == 0, name
        for g, o in zip(logs, ref.log):
            compare_logs(g, o, 1e-4)
        assert rel_l2(z.cpu().numpy(), ref.z) <= TOL_F32, name
