"""Benchmark of the WorldDynCache rollout hot path on one MI355X.

One step = one exact denoising step of the 13B-shaped world model through the
C ABI, i.e. every stage of the hot path: pass-1 lift statistics and the
surrogate candidate (retrieval, lifted evolution, kernel observation), the
risk proxy and decision, the full DiT forward F_theta (20 dual-stream + 40
single-stream blocks, 67,320 video + 256 text tokens, D = 3072, 24 x 128
heads), the Euler step Psi with the counterfactual defect, calibration and the
bank insert. Weights are random-initialised on the device; inputs are seeded
synthetic tensors resident in HBM before timing starts.

Prints one JSON line. ``value`` is the DiT-forward throughput (algorithmic
24*N*D^2 + 4*N^2*D FLOPs per block divided by the measured step time).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 matrix-core peak
PEAK_HBM_GBS = 8000.0
# HBM traffic per attention call of the dominant kernel from two rocprofv3
# --pmc passes (FETCH_SIZE x 2.000 + WRITE_SIZE x 1.000, scale factors from a
# 1 GiB device copy; profiles/attention_13b_hbm_traffic.md): the attention
# kernel plus the combine launch of its split last round. Valid only for the
# kernel version named here; set to None whenever that kernel changes.
MEASURED_TRAFFIC = {"k_attn_bf16_ppr3<128>": 9.386e9}
ATTN_KERNEL = {128: "k_attn_bf16_ppr3<128>", 64: "k_attn_bf16_ppr3<64>"}   # default bf16 kernel by head size
METRIC = "DiT fwd TFLOP/s (% bf16 MFMA peak) + denoising steps/s at 13B shape"
# Risk thresholds (Eq. (10)) of the measured rollouts, one per workload, for the
# device random weights of seed 1234 and the seeded inputs: the centre of the
# threshold range whose risk-controlled schedule makes the paper's exact-call
# ratio for that model class (Sec. 5.1: 20% for the 13B shape, 47% for the 5B
# shape), found from the R_cand values these rollouts log. The rollout reports
# the exact calls it actually made.
RISK_TAU = {"13b": 0.26606899, "5b": 0.18634464}
TARGET_EXACT_RATIO = {"13b": 0.20, "5b": 0.47}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="13b", choices=["13b", "5b", "mid", "tiny"])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline leg")
    ap.add_argument("--surrogate-steps", type=int, default=20)
    ap.add_argument("--no-surrogate", action="store_true", help="skip the standalone surrogate-kernel leg")
    ap.add_argument("--no-batch", action="store_true", help="skip the batched-rollout leg")
    ap.add_argument("--no-rollout", action="store_true",
                    help="skip the measured risk-controlled rollout of the workload (cfg.steps denoising steps)")
    ap.add_argument("--periodic-rollout", action="store_true",
                    help="also time a rollout with periodic placement (exact when k mod 5 == 0)")
    ap.add_argument("--no-stress", action="store_true",
                    help="skip the 118,800-token legs (attention alone and one single-stream block)")
    ap.add_argument("--surrogate-only", action="store_true",
                    help="run only the surrogate-kernel leg (16x33x90x160 latent) and print its JSON")
    ap.add_argument("--stress-only", action="store_true",
                    help="run only the 118,800-token legs (attention alone, one single-stream block) and print "
                         "their JSON")
    ap.add_argument("--no-5b", action="store_true",
                    help="skip the 5B-shaped exact steps and risk-controlled rollout")
    ap.add_argument("--no-library", action="store_true",
                    help="skip the same-box comparison with torch's attention and F.linear")
    ap.add_argument("--library-only", action="store_true",
                    help="run only that comparison (on the workload's shapes) and print its JSON")
    ap.add_argument("--copy-probe", type=int, default=0,
                    help="also run one plain device copy of this many bytes (hardware-counter calibration)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(cfg, rows: int = 64):
    """The oracle on host cores: one block of the workload at its real token count,
    keys/values for every token, queries and the rest for ``rows`` sampled rows."""
    import numpy as np

    import synth
    from oracle import dit
    blk = cfg.n_blocks - 1                      # a single-stream block for the 13B shape
    pre = synth.block_prefix(cfg, blk)
    W = synth.gen_weights(cfg, names=[pre])
    x = synth.gen_block_input(cfg)
    c = synth.gen_cemb(cfg)
    sel = np.linspace(0, cfg.n_tokens - 1, rows).astype(np.int64)
    t0 = time.perf_counter()
    dit.block_forward(W, cfg, blk, x, c, rows=sel)
    dt = time.perf_counter() - t0
    n, d = cfg.n_tokens, cfg.hidden
    f = cfg.mlp_ratio * d
    kind = dit.block_kind(cfg, blk)
    # algorithmic FLOPs of what was evaluated: K,V projections for all tokens,
    # Q/attention/output/MLP for the sampled rows
    flops = 2.0 * n * d * 2 * d + 2.0 * rows * d * d + 4.0 * rows * n * d
    flops += 2.0 * rows * d * f + 2.0 * rows * (d + f) * d if kind == "single" else 2.0 * rows * d * d * 9
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": min(threads, os.cpu_count() or 1),
            "kind": "oracle", "seconds": dt,
            "sample": f"one {kind} block of the {cfg.name} workload in float64: keys/values for all {n} tokens, "
                      f"queries/attention/MLP for {rows} sampled rows ({flops / 1e12:.2f} TFLOP)"}


def cpu_extra(cfg, base):
    """More of the oracle on host cores: the full forward of ``cfg`` extrapolated
    from the sampled block's rate (labelled), one whole forward of the mid
    workload (8 blocks, 2,688 tokens) with its 20-step all-exact rollout
    extrapolated, and the surrogate and risk arithmetic on the 16x33x90x160
    latent with a full bank of 4 (a short replay rollout)."""
    import numpy as np

    import synth
    from oracle import dit
    from oracle import params as P
    from oracle import rollout as ro
    out = {}
    full = cfg.flops_per_forward() / (base["value"] * 1e12)
    out["full_forward_extrapolated"] = {
        "seconds": round(full, 1), "steps_per_s_all_exact": round(1.0 / full, 6),
        "note": f"extrapolated, not measured: {cfg.flops_per_forward() / 1e12:.0f} TFLOP of the {cfg.name} forward "
                f"at the sampled block's {base['value']:.3f} TFLOP/s"}
    mid = synth.get_config("mid")
    W = synth.gen_weights(mid)
    inp = synth.gen_inputs(mid)
    t0 = time.perf_counter()
    dit.dit_forward(W, mid, inp["z_T"], 1.0, inp["cond"])
    dt = time.perf_counter() - t0
    out["mid_forward"] = {"seconds": round(dt, 2), "tflops": round(mid.flops_per_forward() / dt / 1e12, 4),
                          "rollout_20_steps_all_exact_extrapolated_s": round(20 * dt, 1),
                          "note": "one measured float64 forward of the mid workload; the rollout figure is 20x it"}
    del W
    st = synth.get_config("stress")
    steps, mask = 6, [0, 0, 0, 0, 1, 1]
    vel = synth.gen_replay_velocities(st, steps)
    z0 = synth.gen_inputs(st)["z_T"]
    t0 = time.perf_counter()
    res = ro.rollout(ro.replay_denoiser(vel), z0, steps, P.DEFAULTS, mode="forced", forced=mask)
    dt = time.perf_counter() - t0
    out["surrogate_risk_16x33x90x160"] = {
        "ms_per_step": round(dt / steps * 1e3, 1), "steps": steps, "schedule": res.schedule,
        "note": "mean per step of a float64 replay rollout (recorded velocities): 4 exact steps fill the bank, "
                "then 2 surrogate steps read all 4 records; every step lifts the latent, builds the candidate "
                "and evaluates the risk proxy"}
    return out


def hbm_entry(ms, launches, nbytes):
    """Average launch time and achieved algorithmic bandwidth of one HBM-bound kernel class."""
    if not launches:
        return None
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"launches": launches, "ms_avg": round(ms / launches, 4), "bytes_per_launch": round(nbytes / launches),
            "GB/s": round(gbs, 1), "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 3)}


def surrogate_leg(wdc, synth, torch, dev, steps=24):
    """The surrogate and risk kernels alone on the largest latent (16x33x90x160
    float32) with a bank of 4 records: one replay rollout (exact every 4th step,
    recorded velocities standing in for F_theta), then the pass-1 statistics
    kernel on its own through the step-by-step entry point."""
    cfg = synth.get_config("stress")
    ctx = wdc.Context(cfg, device=str(dev), allocate_weights=False)
    st = ctx.new_state()
    gen = torch.Generator(device=dev).manual_seed(cfg.seed)
    lat = tuple(cfg.latent)
    z0 = torch.randn(lat, generator=gen, device=dev)
    base = torch.randn(lat, generator=gen, device=dev)
    vel = torch.empty((steps,) + lat, device=dev)
    for k in range(steps):
        vel[k] = base + 0.3 * torch.randn(lat, generator=gen, device=dev)
    mask = [0 if k % 4 == 0 else 1 for k in range(steps)]
    z = z0.clone()
    ctx.rollout(st, z, steps, mode=wdc.MODE_FORCED, forced=mask, replay_v=vel)    # warm-up
    z.copy_(z0)
    torch.cuda.synchronize()
    ctx.set_timing(True)
    t0 = time.perf_counter()
    sched, logs = ctx.rollout(st, z, steps, mode=wdc.MODE_FORCED, forced=mask, replay_v=vel)
    wall = time.perf_counter() - t0
    tm = ctx.timing()
    ctx.set_timing(False)
    # pass 1 alone (the rollout emits it from the observation / epilogue kernels)
    zhat = torch.empty_like(z)
    ctx.set_timing(True)
    step_ms = []
    for i in range(20):
        t1 = time.perf_counter()
        ctx.surrogate_step(st, z, steps - 1, steps, zhat)
        ctx.risk_update(st, wdc.PRE_DECISION, steps - 1, steps)
        step_ms.append((time.perf_counter() - t1) * 1e3)
    tp = ctx.timing()
    ctx.set_timing(False)
    n_sur = sum(sched)
    res = {"workload": f"latent {'x'.join(map(str, cfg.latent))} float32 ({cfg.numel} elements), bank of 4; "
                       f"replay rollout of {steps} steps, exact every 4th ({steps - n_sur} exact, {n_sur} surrogate)",
           "observe": hbm_entry(*tm["observe"]), "exact_post": hbm_entry(*tm["exact_post"]),
           "stats": hbm_entry(*tp["stats"]),
           "rollout_ms_per_step": round(wall / steps * 1e3, 3),
           "surrogate_step_ms_median": round(float(sorted(step_ms)[len(step_ms) // 2]), 3),
           "note": "bytes = each input read once + each output written once; rollout time includes one "
                   "host synchronisation per step for the float64 controller"}
    del ctx, st, z, z0, base, vel, zhat
    torch.cuda.empty_cache()
    return res


def rollout_leg(wdc, cfg, ctx, inp, torch, dev, tau=None, period=5):
    """One whole rollout of cfg.steps denoising steps through wdc_rollout, timed
    end to end (every exact step's F_theta, every candidate, decision and host
    synchronisation). With ``tau``: the risk controller of Eq. (9)-(10) at that
    threshold; without: periodic placement, exact where k mod period == 0 and
    the lifted surrogate elsewhere whenever it is available."""
    p = wdc.default_params(tau_risk=tau) if tau is not None else wdc.default_params(period=period)
    rctx = wdc.Context(cfg, params=p, device=str(dev), allocate_weights=False)
    rctx.bind_weights(ctx.weights)                              # same weights, bound to the new context
    st = rctx.new_state()
    z = torch.from_numpy(inp["z_T"]).to(dev)
    dv = {k: rctx.to_device(inp[k]) if k in inp else None for k in ("cond", "text", "cam")}
    mode = wdc.MODE_RISK if tau is not None else wdc.MODE_PERIODIC
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    sched, logs = rctx.rollout(st, z, cfg.steps, dv["cond"], dv["text"], dv["cam"], mode=mode)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    n_exact = len(sched) - sum(sched)
    res = {"steps": cfg.steps, "exact_calls": n_exact, "exact_ratio": round(n_exact / cfg.steps, 3),
           "seconds": round(dt, 2), "denoising_steps_per_s": round(cfg.steps / dt, 3),
           "schedule": "".join("S" if s else "E" for s in sched),
           "finite": bool(torch.isfinite(z).all())}
    if tau is not None:
        res["placement"] = f"risk controller, tau = {tau:.6g}"
        res["min_relative_margin"] = round(min(l["margin"] for l in logs if l["available"]), 4)
    else:
        res["placement"] = f"periodic, exact when k mod {period} == 0 (surrogate elsewhere when available)"
    del rctx, st, z
    return res


def second_workload_leg(wdc, synth, torch, dev, name="5b", steps=3):
    """The other model class of the paper's generation experiments (the 5B shape:
    30 sequential blocks over the joint sequence, D = 3,072, 48 x 64 heads,
    17,550 video + 226 text tokens): exact denoising steps timed as in the main measurement (one
    warm-up step, then ``steps`` steps: candidate, risk decision, F_theta, Psi,
    counterfactual and insert), with the attention and GEMM classes timed by
    the library's HIP events, then one measured risk-controlled rollout at the
    threshold giving that class's exact-call ratio (Sec. 5.1: 47%)."""
    cfg = synth.get_config(name)
    ctx = wdc.Context(cfg, device=str(dev))
    ctx.init_random_weights(seed=1234, std=0.02)
    st = ctx.new_state()
    inp = synth.gen_inputs(cfg)
    dv = {k: ctx.to_device(inp[k]) if k in inp else None for k in ("cond", "text", "cam")}
    zb = [torch.from_numpy(inp["z_T"]).to(dev), None]
    zb[1] = torch.empty_like(zb[0])
    zhat, v = torch.empty_like(zb[0]), torch.empty_like(zb[0])
    S = cfg.steps

    def exact_step(k, cur):
        zc, zn = zb[cur], zb[cur ^ 1]
        ctx.surrogate_step(st, zc, k, S, zhat)
        ctx.risk_update(st, wdc.PRE_DECISION, k, S)
        t, tn = (S - k) / S, (S - k - 1) / S
        ctx.forward(zc, t, dv["cond"], dv["text"], dv["cam"], out=v)
        ctx.scheduler_step(zc, v, t, tn, out=zn)
        ctx.risk_update(st, wdc.POST_EXACT, k, S, zc, zn)
        return cur ^ 1

    cur = exact_step(0, 0)
    torch.cuda.synchronize()
    ctx.set_timing(True)
    t0 = time.perf_counter()
    for k in range(1, steps + 1):
        cur = exact_step(k, cur)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / steps * 1e3
    tm = ctx.timing()
    ctx.set_timing(False)
    flops = cfg.flops_per_forward()
    a_ms, a_n, a_work = tm["attention"]
    g_ms, g_n, g_work = tm["gemm"]
    out = {"workload": f"{name}-shaped world model: {cfg.n_blocks} sequential blocks, D={cfg.hidden}, "
                       f"{cfg.heads}x{cfg.head_dim} heads, {cfg.n_video} video + {cfg.text_tokens} text tokens, "
                       f"latent {'x'.join(map(str, cfg.latent))}",
           "ms_per_exact_step": round(ms, 2), "tflops": round(flops / (ms / 1e3) / 1e12, 1),
           "pct_bf16_peak": round(100.0 * flops / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 2),
           "attention_ms_avg": round(a_ms / a_n, 3), "attention_tflops": round(a_work / (a_ms / 1e3) / 1e12, 1),
           "linear_tflops": round(g_work / (g_ms / 1e3) / 1e12, 1)}
    if RISK_TAU.get(name) is not None:
        out["rollout_measured"] = rollout_leg(wdc, cfg, ctx, inp, torch, dev, tau=RISK_TAU[name])
        out["rollout_measured"]["target_exact_ratio"] = TARGET_EXACT_RATIO[name]
    del ctx, st, zb, zhat, v, dv
    torch.cuda.empty_cache()
    return out


def stress_leg(wdc, synth, torch, dev, reps=3):
    """The 118,800-token workload (33 x 45 x 80 tokens, 24 x 128 heads): attention
    alone on random Q, K, V ~ N(0, 1) (4 N^2 D = 173.4 TFLOP per launch), then
    one whole single-stream block on a random residual stream (24 N D^2 + 4 N^2 D
    = 200.3 TFLOP), each timed with HIP events on the library's stream."""
    cfg = synth.get_config("stress")
    ctx = wdc.Context(cfg, device=str(dev))
    ctx.init_random_weights(seed=99, std=0.02)
    n, h, hd = cfg.n_tokens, cfg.heads, cfg.head_dim
    npad = ctx.attn_pad(n)
    gen = torch.Generator(device=dev).manual_seed(cfg.seed)
    def rnd():
        x = torch.zeros((h, npad, hd), dtype=torch.bfloat16, device=dev)
        x[:, :n] = torch.randn((h, n, hd), generator=gen, device=dev).to(torch.bfloat16)
        return x
    q, k = rnd(), rnd()
    vt = torch.zeros((h, hd, npad), dtype=torch.bfloat16, device=dev)
    vt[:, :, :n] = torch.randn((h, hd, n), generator=gen, device=dev).to(torch.bfloat16)
    o = torch.empty((n, h * hd), dtype=torch.bfloat16, device=dev)
    ctx.attention(q, k, vt, n, o, h * hd)                        # warm-up
    ctx.set_timing(True)
    for _ in range(reps):
        ctx.attention(q, k, vt, n, o, h * hd)
    tm = ctx.timing()
    ctx.set_timing(False)
    a_ms, a_n, a_work = tm["attention"]
    att = {"launches": a_n, "ms_avg": round(a_ms / a_n, 3), "tflop_per_launch": round(a_work / a_n / 1e12, 2),
           "tflops": round(a_work / (a_ms / 1e3) / 1e12, 1),
           "frac_bf16_peak": round(a_work / (a_ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "finite": bool(torch.isfinite(o).all())}
    del q, k, vt, o
    x0 = torch.randn((n, cfg.hidden), generator=gen, device=dev)
    c = torch.randn((cfg.hidden,), generator=gen, device=dev)
    x = x0.clone()
    ctx.block_forward(0, x, c)                                   # warm-up
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    times = []
    for _ in range(reps):
        x.copy_(x0)
        ev[0].record()
        ctx.block_forward(0, x, c)
        ev[1].record()
        torch.cuda.synchronize()
        times.append(ev[0].elapsed_time(ev[1]))
    blk_ms = float(sorted(times)[len(times) // 2])
    flops = cfg.flops_per_forward()
    blk = {"ms_median": round(blk_ms, 3), "tflop": round(flops / 1e12, 2),
           "tflops": round(flops / (blk_ms / 1e3) / 1e12, 1),
           "frac_bf16_peak": round(flops / (blk_ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
           "finite": bool(torch.isfinite(x).all())}
    del ctx, x, x0, c
    torch.cuda.empty_cache()
    return {"workload": f"{n} tokens (latent {'x'.join(map(str, cfg.latent))}, patch 1x2x2), {h}x{hd} heads, D={cfg.hidden}",
            "attention_alone": att, "single_block": blk}


def library_leg(wdc, cfg, torch, dev, reps=3):
    """Same-box context for the two dominant kernels: this library's attention
    and plain bf16 product (bias add, no fused epilogue) against torch's
    scaled_dot_product_attention (flash backend) and F.linear on the same
    shapes and inputs, all timed with events on the current stream (the
    library's stream). The library numbers are the product path; torch's are
    context, not a target."""
    import torch.nn.functional as F
    ctx = wdc.Context(cfg, device=str(dev), allocate_weights=False)
    gen = torch.Generator(device=dev).manual_seed(cfg.seed + 7)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(reps):
            fn()
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / reps

    def entry(flop, ms_lib, ms_torch, err):
        return {"ms": round(ms_lib, 3), "tflops": round(flop / ms_lib / 1e9, 1),
                "torch_ms": round(ms_torch, 3) if ms_torch else None,
                "torch_tflops": round(flop / ms_torch / 1e9, 1) if ms_torch else None,
                "speedup_vs_torch": round(ms_torch / ms_lib, 3) if ms_torch else None,
                "rel_l2_vs_torch": float(f"{err:.2e}") if err is not None else None}

    out = {}
    n, h, hd = cfg.n_tokens, cfg.heads, cfg.head_dim
    npad = ctx.attn_pad(n)
    q = torch.zeros((h, npad, hd), dtype=torch.bfloat16, device=dev)
    k, v = torch.zeros_like(q), torch.zeros_like(q)
    for x in (q, k, v):
        x[:, :n] = torch.randn((h, n, hd), generator=gen, device=dev).to(torch.bfloat16)
    # V^T with the key order the kernel takes: within each group of 16 keys,
    # key j sits at column j with bits 2 and 3 swapped
    j = torch.arange(npad, device=dev)
    col = (j & ~12) | ((j & 4) << 1) | ((j & 8) >> 1)
    vt = torch.empty((h, hd, npad), dtype=torch.bfloat16, device=dev)
    vt[:, :, col] = v.transpose(1, 2)
    o = torch.empty((n, h * hd), dtype=torch.bfloat16, device=dev)
    ms_lib = timed(lambda: ctx.attention(q, k, vt, n, o, h * hd))
    q4, k4, v4 = (x[:, :n].unsqueeze(0) for x in (q, k, v))
    ms_t, err, note = None, None, None
    try:
        with torch.nn.attention.sdpa_kernel(torch.nn.attention.SDPBackend.FLASH_ATTENTION):
            ms_t = timed(lambda: F.scaled_dot_product_attention(q4, k4, v4))
            ref = F.scaled_dot_product_attention(q4, k4, v4)[0].transpose(0, 1).reshape(n, h * hd).float()
        err = ((o.float() - ref).norm() / ref.norm()).item()
        del ref
    except Exception as e:  # a torch build without the flash backend: report the library alone
        note = f"torch flash attention unavailable: {str(e)[:100]}"
    out["attention"] = entry(4.0 * n * n * hd * h, ms_lib, ms_t, err)
    if note:
        out["attention"]["note"] = note
    del q, k, v, vt, o, q4, k4, v4
    torch.cuda.empty_cache()
    d, f = cfg.hidden, cfg.mlp_ratio * cfg.hidden
    for name, (nn_, kk) in (("qkv", (3 * d, d)), ("mlp_in", (f, d)), ("single_out", (d, d + f)),
                            ("mlp_out", (d, f)), ("attn_out", (d, d))):
        a = torch.randn((n, kk), generator=gen, device=dev).to(torch.bfloat16)
        w = (0.02 * torch.randn((nn_, kk), generator=gen, device=dev)).to(torch.bfloat16)
        b = (0.1 * torch.randn((nn_,), generator=gen, device=dev)).to(torch.bfloat16)
        c = torch.empty((n, nn_), dtype=torch.bfloat16, device=dev)
        ms_lib = timed(lambda: ctx.linear(a, w, b, c, n, nn_, kk))
        ms_t = timed(lambda: F.linear(a, w, b))
        ref = F.linear(a, w, b).float()
        err = ((c.float() - ref).norm() / ref.norm()).item()
        out[f"linear_{name}"] = dict(entry(2.0 * n * nn_ * kk, ms_lib, ms_t, err), shape=[n, nn_, kk])
        del a, w, b, c, ref
        torch.cuda.empty_cache()
    del ctx
    torch.cuda.empty_cache()
    return out


def batched_leg(wdc, synth, torch, dev, steps=20, batches=(1, 8)):
    """Throughput of batched rollouts on the mid workload (8 blocks, D = 1024, 2,688
    tokens, bf16): B independent all-exact rollouts of `steps` denoising steps, F_theta
    evaluated once per step for the whole batch, against B = 1."""
    import dataclasses
    cfg = synth.get_config("mid")
    bmax = max(batches)
    ctx = wdc.Context(cfg, device=str(dev), max_batch=bmax)
    ctx.init_random_weights(seed=7, std=0.02)
    inp = [synth.gen_inputs(dataclasses.replace(cfg, seed=cfg.seed + b)) for b in range(bmax)]
    z0 = [torch.from_numpy(i["z_T"]).to(dev) for i in inp]
    cond = [ctx.to_device(i["cond"]) for i in inp]
    states = [ctx.new_state() for _ in range(bmax)]
    out = {"workload": f"mid: {cfg.n_blocks} blocks, D={cfg.hidden}, {cfg.n_tokens} tokens, latent "
                       f"{'x'.join(map(str, cfg.latent))}; all-exact rollouts of {steps} steps", "runs": []}
    base = None
    for B in batches:
        zs = [z.clone() for z in z0[:B]]
        ctx.rollout_batch(states[:B], zs, steps, cond[:B], mode=wdc.MODE_ALL_EXACT)      # warm-up
        zs = [z.clone() for z in z0[:B]]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ctx.rollout_batch(states[:B], zs, steps, cond[:B], mode=wdc.MODE_ALL_EXACT)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        sps = B * steps / dt
        base = base or sps
        out["runs"].append({"batch": B, "seconds": round(dt, 4), "denoising_steps_per_s": round(sps, 1),
                            "tflops": round(B * steps * cfg.flops_per_forward() / dt / 1e12, 1),
                            "speedup_vs_batch1": round(sps / base, 2)})
    del ctx, states, z0, cond
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the multi-GPU path is not built", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2608_01845_amd as wdc
    import synth

    cfg = synth.get_config(args.workload)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.surrogate_only:
        print(json.dumps({"surrogate_kernels": surrogate_leg(wdc, synth, torch, dev)}), flush=True)
        return
    if args.stress_only:
        print(json.dumps({"stress_118800": stress_leg(wdc, synth, torch, dev)}), flush=True)
        return
    if args.library_only:
        print(json.dumps({"library_comparison": library_leg(wdc, cfg, torch, dev)}), flush=True)
        return
    S = cfg.steps
    log(f"workload {cfg.name}: {cfg.n_blocks} blocks, N={cfg.n_tokens}, D={cfg.hidden}, {cfg.heads}x{cfg.head_dim}")
    ctx = wdc.Context(cfg, device="cuda:0")
    ctx.init_random_weights(seed=1234, std=0.02)
    st = ctx.new_state()
    inp = synth.gen_inputs(cfg)
    z = torch.from_numpy(inp["z_T"]).to(dev)
    cond = ctx.to_device(inp["cond"]) if "cond" in inp else None
    text = ctx.to_device(inp["text"]) if "text" in inp else None
    cam = ctx.to_device(inp["cam"]) if "cam" in inp else None
    zbuf = [z, torch.empty_like(z)]
    zhat = torch.empty_like(z)
    v = torch.empty_like(z)
    torch.cuda.synchronize()

    def exact_step(k, cur):
        if k and k % S == 0:
            st.reset()            # the schedule's S steps are used up: a new rollout
        k %= S
        zc, zn = zbuf[cur], zbuf[cur ^ 1]
        ctx.surrogate_step(st, zc, k, S, zhat)
        ctx.risk_update(st, wdc.PRE_DECISION, k, S)
        t, tn = (S - k) / S, (S - k - 1) / S
        ctx.forward(zc, t, cond, text, cam, out=v)
        ctx.scheduler_step(zc, v, t, tn, out=zn)
        ctx.risk_update(st, wdc.POST_EXACT, k, S, zc, zn)
        return cur ^ 1

    cur, k = 0, 0
    for _ in range(args.warmup):
        t0 = time.perf_counter()
        cur = exact_step(k, cur)
        torch.cuda.synchronize()
        k += 1
        log(f"warmup step {k} {time.perf_counter() - t0:.2f}s")
    ctx.set_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        cur = exact_step(k, cur)
        k += 1
        torch.cuda.synchronize()
        log(f"timed step {i + 1}/{args.steps} done ({time.perf_counter() - t0:.2f}s)")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    # device memory of the exact steps: the library's weights, workspace and
    # rollout state all come from torch allocations
    free_b, total_b = torch.cuda.mem_get_info(dev)
    memory = {"peak_allocated_gb": round(torch.cuda.max_memory_allocated(dev) / 1e9, 2),
              "device_used_gb": round((total_b - free_b) / 1e9, 2), "device_total_gb": round(total_b / 1e9, 1)}
    timing = ctx.timing()
    ctx.set_timing(False)
    ms_step = elapsed / args.steps * 1e3
    fwd_flops = cfg.flops_per_forward()
    tflops = fwd_flops / (ms_step / 1e3) / 1e12

    # surrogate-step cost (candidate + risk), the other branch of the rollout
    sur_ms = []
    for i in range(args.surrogate_steps):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        ctx.surrogate_step(st, zbuf[cur], k % S, S, zhat)
        ctx.risk_update(st, wdc.PRE_DECISION, k % S, S)
        torch.cuda.synchronize()
        sur_ms.append((time.perf_counter() - t1) * 1e3)
    sur_med = float(np.median(sur_ms))

    # roofline of the dominant kernel (attention: 4 N^2 D per block), from the
    # library's HIP events on its own stream over the timed steps
    att_ms, att_n, att_work = timing["attention"]
    att_avg_ms = att_ms / max(att_n, 1)
    att_tflops = att_work / (att_ms / 1e3) / 1e12 if att_n else None
    gemm_ms, gemm_n, gemm_work = timing["gemm"]
    gemm_tflops = gemm_work / (gemm_ms / 1e3) / 1e12 if gemm_ms else None
    norm_ms, norm_n, norm_work = timing["norm"]

    exact_ratio = TARGET_EXACT_RATIO.get(cfg.name, 0.20)
    n_exact = round(exact_ratio * S)
    derived_rollout_s = (n_exact * ms_step + (S - n_exact) * sur_med) / 1e3

    out = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded latents/conditions, device random-init weights)",
        "config": {
            "workload": f"{cfg.name}-shaped world model: {cfg.n_dual} dual + {cfg.n_single} single + {cfg.n_seq} "
                        f"sequential blocks, D={cfg.hidden}, {cfg.heads}x{cfg.head_dim} heads, "
                        f"{cfg.n_video} video + {cfg.text_tokens} text tokens, latent {'x'.join(map(str, cfg.latent))}; "
                        f"step = one exact denoising step (candidate + risk + F_theta + Psi + counterfactual + insert)",
            "global_batch": 1, "seq_len": cfg.n_tokens, "parallelism": "none (1 GPU)"},
        "pct_bf16_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 2),
        "denoising_steps_per_s_exact": round(1e3 / ms_step, 4),
        "surrogate_step_ms": round(sur_med, 3),
        "memory": memory,
        "derived_rollout_estimate": {"steps": S, "exact_ratio": exact_ratio, "seconds": round(derived_rollout_s, 2),
                                     "steps_per_s": round(S / derived_rollout_s, 3),
                                     "note": "arithmetic on the measured exact-step and surrogate-step times, "
                                             "not a measurement; rollout_measured is the measured rollout"},
        "kernels": {"attention_ms_avg": round(att_avg_ms, 3), "attention_launches": att_n,
                    "attention_tflops": round(att_tflops, 1) if att_tflops else None,
                    "gemm_ms_total": round(gemm_ms, 1), "gemm_launches": gemm_n,
                    "linear_tflops": round(gemm_tflops, 1) if gemm_tflops else None,
                    "layernorm_modulate": hbm_entry(norm_ms, norm_n, norm_work),
                    # query blocks of 256 per head over all keys, and the key ranges each
                    # block of the last, partial dispatch round runs as (1: no split)
                    "attention_plan": dict(zip(("query_blocks_over_all_keys", "key_ranges_of_the_rest"),
                                               ctx.attention_plan(cfg.n_tokens)))},
        "roofline": {"bound": "mfma",
                     # one attention call: the kernel, plus the combine launch when its last
                     # dispatch round runs as key-range splits
                     "kernel": ATTN_KERNEL.get(cfg.head_dim) + (
                         f" + k_attn_combine<{cfg.head_dim}>" if ctx.attention_plan(cfg.n_tokens)[1] > 1 else ""),
                     "achieved": round(att_tflops, 1) if att_tflops else None,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(att_tflops / PEAK_BF16_TFLOPS, 4) if att_tflops else None,
                     "traffic": MEASURED_TRAFFIC.get(ATTN_KERNEL.get(cfg.head_dim)) if args.workload == "13b" else None,
                     "traffic_unit": "bytes per attention call (attention kernel + combine)"},
    }
    if not args.no_rollout and RISK_TAU.get(cfg.name) is not None:
        log(f"measured risk-controlled rollout ({S} steps) ...")
        t0 = time.perf_counter()
        out["rollout_measured"] = rollout_leg(wdc, cfg, ctx, inp, torch, dev, tau=RISK_TAU[cfg.name])
        out["rollout_measured"]["target_exact_ratio"] = TARGET_EXACT_RATIO[cfg.name]
        out["denoising_steps_per_s_rollout"] = out["rollout_measured"]["denoising_steps_per_s"]
        log(f"rollout done ({time.perf_counter() - t0:.1f}s, {out['rollout_measured']['exact_calls']} exact)")
    if args.periodic_rollout:
        log("periodic-placement rollout ...")
        out["rollout_periodic"] = rollout_leg(wdc, cfg, ctx, inp, torch, dev)
    del ctx, st, z, zbuf, zhat, v, cond, text, cam
    torch.cuda.empty_cache()
    if not args.no_5b and args.workload == "13b":
        log("5B-shaped exact steps and risk-controlled rollout ...")
        out["workload_5b"] = second_workload_leg(wdc, synth, torch, dev)
    if not args.no_stress:
        log("118,800-token attention and single block ...")
        out["stress_118800"] = stress_leg(wdc, synth, torch, dev)
    if not args.no_surrogate:
        out["surrogate_kernels"] = surrogate_leg(wdc, synth, torch, dev)
    if not args.no_library:
        log("same-box comparison with torch's attention and products ...")
        out["library_comparison"] = library_leg(wdc, cfg, torch, dev)
    if not args.no_batch:
        log("batched rollouts (mid workload) ...")
        out["batched_rollout"] = batched_leg(wdc, synth, torch, dev)
    if args.copy_probe > 0:
        src = torch.empty(args.copy_probe // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_probe_bytes"] = args.copy_probe
        del src, dst
    if not args.no_cpu:
        log("CPU oracle baseline ...")
        out["cpu_baseline"] = cpu_baseline(cfg)
        log(f"CPU oracle baseline done ({out['cpu_baseline']['seconds']:.1f}s)")
        out["cpu_baseline"]["extra"] = cpu_extra(cfg, out["cpu_baseline"])
        log("CPU oracle extra legs done")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
