"""The allocation-free surrogate step (wdc_surrogate_step_noalloc) against
wdc_surrogate_step through the C ABI: two states driven through the same
steps, one per entry point, must give bit-identical candidates and logs. Two
latents in a row, the second smaller, so the fixed scratch array holds the
first call's contents when the second starts."""
import math

import numpy as np
import pytest

import synth
from tests.gpu_util import small_cfg, torch_cuda

pytestmark = pytest.mark.gpu


def _same(a: dict, b: dict):
    assert a.keys() == b.keys()
    for key in a:
        x, y = np.asarray(a[key], dtype=np.float64), np.asarray(b[key], dtype=np.float64)
        assert np.array_equal(x, y, equal_nan=True), (key, a[key], b[key])


def _drive(cfg, steps=6):
    """Steps 0..steps-1 with exact commits at even steps and surrogate commits at
    odd ones (when available), on one state per entry point."""
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    ctx = wdc.Context(cfg, allocate_weights=False)
    vel = torch.from_numpy(synth.gen_replay_velocities(cfg, steps)).cuda()
    z0 = torch.from_numpy(synth.gen_inputs(cfg)["z_T"]).cuda()
    s_ref, s_na = ctx.new_state(), ctx.new_state()
    z = z0.clone()
    zh_ref, zh_na = torch.full_like(z, 7.0), torch.full_like(z, -7.0)
    observed = 0
    for k in range(steps):
        log_ref = ctx.surrogate_step(s_ref, z, k, steps, zh_ref)
        log_na = ctx.surrogate_step_noalloc(s_na, z, k, steps, zh_na)
        _same(log_ref, log_na)
        if log_ref["bank"]:
            assert torch.equal(zh_ref, zh_na)
            observed += 1
        d_ref = ctx.risk_update(s_ref, wdc.PRE_DECISION, k, steps)
        d_na = ctx.risk_update(s_na, wdc.PRE_DECISION, k, steps)
        _same(d_ref, d_na)
        if k % 2 == 1 and d_ref["available"]:
            for s in (s_ref, s_na):
                ctx.risk_update(s, wdc.POST_SURROGATE, k, steps)
            z = zh_ref.clone()
        else:
            zn = ctx.scheduler_step(z, vel[k], (steps - k) / steps, (steps - k - 1) / steps)
            _same(ctx.risk_update(s_ref, wdc.POST_EXACT, k, steps, z, zn),
                  ctx.risk_update(s_na, wdc.POST_EXACT, k, steps, z, zn))
            z = zn
    assert observed >= steps - 1 and math.isfinite(float(z.abs().sum()))
    return ctx.cfg.numel


def test_noalloc_surrogate_step_equals_allocating_one_on_two_latents_in_a_row():
    big = _drive(synth.get_config("mid"))
    # second latent smaller, with segment starts that are not 16-byte aligned
    small = _drive(small_cfg("f32"))
    assert small < big


def test_noalloc_surrogate_step_rejects_bad_arguments():
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    cfg = synth.get_config("tiny")
    ctx = wdc.Context(cfg, allocate_weights=False)
    st = ctx.new_state()
    z = torch.zeros(cfg.latent, device="cuda")
    with pytest.raises(wdc.WdcError):
        ctx.surrogate_step_noalloc(st, z, 8, 8, torch.empty_like(z))       # k outside 0..S-1
