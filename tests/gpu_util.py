"""Shared helpers of the GPU parity tests (seeded inputs, tolerances, contexts)."""
from __future__ import annotations

import os

import numpy as np
import pytest

import synth

# Tolerances: relative L2 error per block / kernel and on the final latent.
TOL_F32 = 1e-4
TOL_BF16_BLOCK = 2e-2
TOL_BF16_FINAL = 5e-2


def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def row_rel_l2(a, b) -> float:
    """Largest relative L2 error of one row (last axis) over all rows."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    num = np.linalg.norm(a - b, axis=-1)
    den = np.maximum(np.linalg.norm(b, axis=-1), 1e-30)
    return float(np.max(num / den))


def small_cfg(dtype="bf16", head_dim=64, **kw):
    """A small joint-sequence model with all three block kinds, text tokens and a camera vector."""
    heads = 256 // head_dim
    rope = (16, 24, 24) if head_dim == 64 else (16, 56, 56)
    base = dict(name="unit", dtype=dtype, hidden=256, heads=heads, head_dim=head_dim, n_seq=1, n_dual=1,
                n_single=1, cond_dim=64, cam_dim=96, text_tokens=21, text_dim=128, latent=(16, 3, 10, 14),
                patch=(1, 2, 2), rope=rope, steps=8, seed=11)
    base.update(kw)
    return synth.ModelConfig(**base)


def wdc_params(p):
    """The library's parameter struct holding the oracle parameters ``p``."""
    from dataclasses import fields
    import paper_2608_01845_amd as wdc
    codes = {"surrogate": {"lifted": wdc.SURROGATE_LIFTED, "secant": wdc.SURROGATE_SECANT},
             "observation": {"kernel": wdc.OBS_KERNEL, "linear": wdc.OBS_LINEAR}}
    out = wdc.default_params()
    for f in fields(p):
        v = getattr(p, f.name)
        if f.name in codes:
            v = codes[f.name][v]
        elif isinstance(v, bool):
            v = int(v)
        setattr(out, f.name, v)
    return out


def context(cfg, weights=True, params=None, fill_tiles=True):
    """A context on cuda:0. fill_tiles=False: GEMM tile size by shape alone
    (products too small to fill one dispatch round of 256 x 256 tiles keep
    those tiles instead of moving to 128 x 128 ones)."""
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    if not fill_tiles:
        os.environ["WDC_FILL_TILES"] = "0"
    try:
        ctx = wdc.Context(cfg, params=params, allocate_weights=weights)
    finally:
        os.environ.pop("WDC_FILL_TILES", None)
    if weights:
        ctx.load_weights(synth.gen_weights(cfg))
    return ctx


def dev_inputs(ctx, cfg):
    inp = synth.gen_inputs(cfg)
    out = {"z_T": ctx.to_device(inp["z_T"], dtype=__import__("torch").float32)}
    for k in ("cond", "text", "cam"):
        out[k] = ctx.to_device(inp[k]) if k in inp else None
    return inp, out


def pick_tau(run, lo=0.0, hi=2.0, target_surrogates=None, margin=1e-3, tries=200, seed=0):
    """A risk threshold whose oracle schedule keeps every decision at least ``margin``
    (relative) away from the threshold: run(tau) -> oracle Result."""
    rng = np.random.default_rng(seed)
    best = None
    for _ in range(tries):
        tau = float(rng.uniform(lo, hi))
        res = run(tau)
        m = min((l.margin for l in res.log if l.available), default=np.inf)
        if m < margin:
            continue
        n_sur = sum(res.schedule)
        if target_surrogates is None or n_sur == target_surrogates:
            return tau, res
        if best is None or abs(n_sur - target_surrogates) < abs(best[1] - target_surrogates):
            best = (tau, n_sur, res)
    if best is None:
        raise RuntimeError("no threshold with a clear margin")
    return best[0], best[2]
