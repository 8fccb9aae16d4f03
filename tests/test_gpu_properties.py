"""Property-based shapes for the two MFMA kernels (GPU): hypothesis draws the
product and sequence sizes (derandomized, so every run draws the same cases)
and each result is compared with the oracle at the tolerances of the fixed
cases in test_gpu_kernels.py: bf16 GEMM 4e-3 relative L2 and 1e-2 per row,
bf16 attention 1e-2 and 3e-2 per row and head; the attention's key-range
split of its last dispatch round is drawn with forced range counts."""
import math
import os

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import synth
from oracle import dit
from tests.gpu_util import context, rel_l2, row_rel_l2, small_cfg, torch_cuda
from tests.test_gpu_kernels import ROW_TOL_ATTN_BF16, ROW_TOL_LINEAR_BF16, _attn_inputs

pytestmark = pytest.mark.gpu

SETTINGS = settings(max_examples=30, deadline=None, derandomize=True, database=None,
                    suppress_health_check=list(HealthCheck))
_ctx = {}


def _cached(key, make):
    if key not in _ctx:
        _ctx[key] = make()
    return _ctx[key]


@SETTINGS
@given(m=st.integers(1, 1300), n_blocks=st.integers(1, 20), k_blocks=st.integers(1, 24), fill=st.booleans(),
       seed=st.integers(0, 2**31 - 1))
def test_linear_bf16_any_shape(m, n_blocks, k_blocks, fill, seed):
    """c = a w^T + b for M in [1, 1300], N a multiple of 64 up to 1280 and K a
    multiple of 64 up to 1536, on either tile rule (products below one dispatch
    round of 256 x 256 tiles on 128 x 128 tiles, or tile size by shape alone)."""
    torch = torch_cuda()
    n, k = 64 * n_blocks, 64 * k_blocks
    cfg = synth.get_config("mid")
    ctx = _cached(("linear", fill), lambda: context(cfg, weights=False, fill_tiles=fill))
    rng = np.random.default_rng(seed)
    a = synth.stored(rng.standard_normal((m, k)), cfg.dtype)
    w = synth.stored(rng.standard_normal((n, k)) * 0.05, cfg.dtype)
    b = synth.stored(rng.standard_normal(n) * 0.1, cfg.dtype)
    out = torch.empty((m, n), dtype=ctx.tdtype, device="cuda")
    ctx.linear(ctx.to_device(a), ctx.to_device(w), ctx.to_device(b), out, m, n, k)
    ref = dit.linear({"l.w": w, "l.b": b}, "l", a.astype(np.float64))
    got = out.float().cpu().numpy()
    err, rerr = rel_l2(got, ref), row_rel_l2(got, ref)
    assert err <= 4e-3 and rerr <= ROW_TOL_LINEAR_BF16, (m, n, k, fill, err, rerr)


@SETTINGS
@given(n=st.integers(1, 1400), head_dim=st.sampled_from([64, 128]), seed=st.integers(0, 2**31 - 1))
def test_attention_bf16_any_length(n, head_dim, seed):
    """softmax(q k^T / sqrt(hd)) v for any sequence length from 1 to 1,400 at
    both head sizes (the small model's 4 or 2 heads)."""
    torch = torch_cuda()
    cfg = small_cfg("bf16", head_dim=head_dim)
    ctx = _cached(("attention", head_dim), lambda: context(cfg, weights=False))
    heads = cfg.heads
    (q, k, v), (qd, kd, vd) = _attn_inputs(ctx, heads, head_dim, n, seed=seed, bf16=True)
    out = torch.zeros((n, heads * head_dim), dtype=torch.bfloat16, device="cuda")
    ctx.attention(qd, kd, vd, n, out, heads * head_dim)
    got = out.float().cpu().numpy()
    ref = dit.attention(q, k, v).transpose(1, 0, 2).reshape(n, heads * head_dim)
    err = rel_l2(got, ref)
    rerr = row_rel_l2(got.reshape(n, heads, head_dim), ref.reshape(n, heads, head_dim))
    assert err <= 1e-2 and rerr <= ROW_TOL_ATTN_BF16, (n, head_dim, err, rerr)


@SETTINGS
@given(n=st.integers(65, 3000), head_dim=st.sampled_from([64, 128]), heads_i=st.integers(0, 2),
       splits=st.integers(2, 8), seed=st.integers(0, 2**31 - 1))
def test_attention_split_round_any_length(n, head_dim, heads_i, splits, seed):
    """The key-range split of the last dispatch round (forced: splits ranges
    whenever a round is partial and the scratch holds them) for lengths 65 to
    3,000 and 4, 8 or 16 heads at hd 64 (2, 4 or 8 at hd 128), sampled query
    rows against the oracle; the plan must have split or have had no partial
    round to split."""
    torch = torch_cuda()
    heads = (4, 8, 16)[heads_i] if head_dim == 64 else (2, 4, 8)[heads_i]

    def make():
        os.environ["WDC_ATTN_SPLITS"] = str(splits)
        try:
            return context(small_cfg("bf16", head_dim=head_dim, heads=heads, hidden=heads * head_dim,
                                     latent=(16, 8, 64, 64)), weights=False)
        finally:
            del os.environ["WDC_ATTN_SPLITS"]
    ctx = _cached(("split", head_dim, heads, splits), make)
    # the plan's rule: whole rounds of heads x qb_main blocks over all keys, the
    # rest as min(splits, key tiles) ranges when the scratch (the workspace's
    # projection area, 3 x hidden bf16 values per model token) holds them
    qb_main, ks = ctx.attention_plan(n)
    nqb, tiles = ctx.attn_pad(n) // 256, (n + 63) // 64
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    g = cus // math.gcd(cus, heads)
    tail = nqb - nqb // g * g
    s_eff = min(splits, tiles)
    tokens = 8 * 32 * 32 + 21
    fits = heads * tail * s_eff * 256 * (head_dim + 2) * 4 <= tokens * 3 * heads * head_dim * 2
    expect = (nqb // g * g, s_eff) if tail and s_eff > 1 and fits else (nqb, 1)
    assert (qb_main, ks) == expect, (qb_main, ks, expect)
    (q, k, v), (qd, kd, vd) = _attn_inputs(ctx, heads, head_dim, n, seed=seed, bf16=True)
    out = torch.zeros((n, heads * head_dim), dtype=torch.bfloat16, device="cuda")
    ctx.attention(qd, kd, vd, n, out, heads * head_dim)
    rng = np.random.default_rng(seed)
    rows = np.unique(np.r_[0:3, rng.integers(0, n, 10), n - 3:n])
    got = out.float().cpu().numpy().reshape(n, heads, head_dim)[rows]
    ref = dit.attention(q[:, rows], k, v).transpose(1, 0, 2)
    err, rerr = rel_l2(got, ref), row_rel_l2(got, ref)
    assert np.isfinite(got).all() and err <= 1e-2 and rerr <= ROW_TOL_ATTN_BF16, (n, head_dim, heads, splits, err, rerr)
