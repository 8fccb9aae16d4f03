"""Kernel-level parity of the HIP path against the oracle (GPU)."""
import math

import numpy as np
import pytest

import synth
from oracle import dit, scheduler
from tests.gpu_util import TOL_F32, context, rel_l2, row_rel_l2, small_cfg, torch_cuda

# per-row bounds next to the whole-tensor ones: no row may carry an error the
# average hides (bf16 output rounding alone is about 2^-9 per element)
ROW_TOL_LINEAR_BF16 = 1e-2
ROW_TOL_ATTN_BF16 = 3e-2

pytestmark = pytest.mark.gpu


def _rng(seed):
    return np.random.default_rng(seed)


def test_scheduler_step_matches_closed_form():
    torch = torch_cuda()
    ctx = context(synth.get_config("tiny"), weights=False)
    rng = _rng(0)
    for n in (1, 1000, 16 * 7 * 32 * 48 + 3):
        z = rng.standard_normal(n).astype(np.float32)
        v = rng.standard_normal(n).astype(np.float32)
        zd, vd = (torch.from_numpy(a).cuda() for a in (z, v))
        out = ctx.scheduler_step(zd, vd, 0.65, 0.6).cpu().numpy()
        ref = scheduler.psi(z, v, 0.65, 0.6)
        assert np.max(np.abs(out - ref)) <= 1e-6 * (1 + np.abs(ref).max())


@pytest.mark.parametrize("fill_tiles", [True, False])
@pytest.mark.parametrize("dtype,m,n,k", [
    ("bf16", 1000, 512, 3072), ("bf16", 600, 768, 1024), ("bf16", 300, 256, 128), ("bf16", 130, 384, 64),
    ("bf16", 37, 64, 64), ("bf16", 700, 64, 1024), ("bf16", 67, 192, 512), ("bf16", 1, 128, 256),
    ("bf16", 700, 2048, 256), ("bf16", 2100, 4096, 128),
    ("f32", 300, 320, 96), ("f32", 5, 64, 256)])
def test_linear_matches_oracle(dtype, m, n, k, fill_tiles):
    """fill_tiles=True: these products fill less than one dispatch round of
    256 x 256 tiles, so those with N % 128 == 0 run on 128 x 128 tiles; False:
    the same products on the tiles their shape alone selects (256 x 256 where
    N % 256 == 0 and M >= 512), so both kernels meet ragged M tails."""
    torch = torch_cuda()
    cfg = synth.get_config("mid" if dtype == "bf16" else "tiny")
    ctx = context(cfg, weights=False, fill_tiles=fill_tiles)
    rng = _rng(m * 7 + n)
    a = synth.stored(rng.standard_normal((m, k)), cfg.dtype)
    w = synth.stored(rng.standard_normal((n, k)) * 0.05, cfg.dtype)
    b = synth.stored(rng.standard_normal(n) * 0.1, cfg.dtype)
    out = torch.empty((m, n), dtype=ctx.tdtype, device="cuda")
    ctx.linear(ctx.to_device(a), ctx.to_device(w), ctx.to_device(b), out, m, n, k)
    ref = dit.linear({"l.w": w, "l.b": b}, "l", a.astype(np.float64))
    got = out.float().cpu().numpy()
    err, rerr = rel_l2(got, ref), row_rel_l2(got, ref)
    print(f"{dtype} {m}x{n}x{k}: rel_l2 {err:.2e}, worst row {rerr:.2e}")
    # bf16: output rounding (2^-9) dominates; f32: accumulation order only
    assert err <= (4e-3 if dtype == "bf16" else TOL_F32), err
    assert rerr <= (ROW_TOL_LINEAR_BF16 if dtype == "bf16" else 10 * TOL_F32), rerr


def test_linear_output_rows_not_16_byte_aligned():
    """bf16 output rows 8-byte but not 16-byte aligned (ldc = n + 4): the
    product would take the 256 x 256 kernels (tile size by shape alone), whose
    staged epilogue stores 16-byte chunks, so it must run on the 128 x 128
    kernels instead. Columns past n stay untouched."""
    torch = torch_cuda()
    cfg = synth.get_config("mid")
    ctx = context(cfg, weights=False, fill_tiles=False)
    m, n, k = 600, 512, 256
    rng = _rng(77)
    a = synth.stored(rng.standard_normal((m, k)), cfg.dtype)
    w = synth.stored(rng.standard_normal((n, k)) * 0.05, cfg.dtype)
    b = synth.stored(rng.standard_normal(n) * 0.1, cfg.dtype)
    out = torch.zeros((m, n + 4), dtype=ctx.tdtype, device="cuda")
    ctx.linear(ctx.to_device(a), ctx.to_device(w), ctx.to_device(b), out, m, n, k, ldc=n + 4)
    got = out.float().cpu().numpy()
    err = rel_l2(got[:, :n], dit.linear({"l.w": w, "l.b": b}, "l", a.astype(np.float64)))
    assert err <= 4e-3, err
    assert np.all(got[:, n:] == 0)


@pytest.mark.parametrize("n", [8192, 9216])
def test_linear_large_product_rectangle_order(n):
    """Products big enough for the XCD-rectangle block order (8 x 4 tiles per
    XCD per dispatch round: 65 M tiles in 9 bands, the last one partial, x 32
    or 36 N tiles), with blocks past the last tile in the final dispatch round.
    Sampled rows, including every row of the partial band, against the oracle;
    the whole output against a float32 product."""
    torch = torch_cuda()
    cfg = synth.get_config("mid")
    ctx = context(cfg, weights=False)
    m, k = 16484, 64
    rng = _rng(2024)
    a = synth.stored(rng.standard_normal((m, k)), cfg.dtype)
    w = synth.stored(rng.standard_normal((n, k)) * 0.05, cfg.dtype)
    b = synth.stored(rng.standard_normal(n) * 0.1, cfg.dtype)
    out = torch.empty((m, n), dtype=ctx.tdtype, device="cuda")
    ctx.linear(ctx.to_device(a), ctx.to_device(w), ctx.to_device(b), out, m, n, k)
    rows = np.unique(np.concatenate([rng.choice(16384, 96, replace=False), np.arange(16384, m)]))
    got = out[torch.from_numpy(rows).cuda()].float().cpu().numpy()
    ref = dit.linear({"l.w": w, "l.b": b}, "l", a[rows].astype(np.float64))
    err, rerr = rel_l2(got, ref), row_rel_l2(got, ref)
    print("rows", len(rows), "rel_l2", err, "worst row", rerr)
    assert err <= 4e-3 and rerr <= ROW_TOL_LINEAR_BF16, (err, rerr)
    # every tile written: the whole output against a float32 torch product of
    # the same (bf16-valued) operands
    full = torch.from_numpy(a).cuda() @ torch.from_numpy(w).cuda().T + torch.from_numpy(b).cuda()
    d = (out.float() - full).norm(dim=1) / full.norm(dim=1)
    print("whole output: worst row", float(d.max()))
    assert float(d.max()) <= ROW_TOL_LINEAR_BF16


def test_linear_long_k_tail_split():
    """A long-K product whose last dispatch round would be thin (9 M tiles x 32
    N tiles = 288 tiles, 32 past the last whole round of 256): the first 2,048
    rows run as 256 x 256 tiles and the last 100 as 128 x 128 tiles (a second
    launch). Sampled rows of the first part and every row of the second against
    the oracle."""
    torch = torch_cuda()
    cfg = synth.get_config("mid")
    ctx = context(cfg, weights=False)
    m, n, k = 2148, 8192, 8192
    rng = _rng(2025)
    a = synth.stored(rng.standard_normal((m, k), dtype=np.float32), cfg.dtype)
    w = synth.stored(rng.standard_normal((n, k), dtype=np.float32) * 0.02, cfg.dtype)
    b = synth.stored(rng.standard_normal(n, dtype=np.float32) * 0.1, cfg.dtype)
    out = torch.empty((m, n), dtype=ctx.tdtype, device="cuda")
    ctx.linear(ctx.to_device(a), ctx.to_device(w), ctx.to_device(b), out, m, n, k)
    rows = np.unique(np.concatenate([rng.choice(2048, 48, replace=False), np.arange(2040, m)]))
    got = out[torch.from_numpy(rows).cuda()].float().cpu().numpy()
    ref = dit.linear({"l.w": w, "l.b": b}, "l", a[rows].astype(np.float64))
    err, rerr = rel_l2(got, ref), row_rel_l2(got, ref)
    print("rows", len(rows), "rel_l2", err, "worst row", rerr)
    assert err <= 4e-3 and rerr <= ROW_TOL_LINEAR_BF16, (err, rerr)


def _attn_inputs(ctx, heads, hd, n, seed, bf16):
    rng = _rng(seed)
    q, k, v = (rng.standard_normal((heads, n, hd)) for _ in range(3))
    if bf16:
        q, k, v = (synth.round_bf16(x).astype(np.float64) for x in (q, k, v))
    return (q, k, v), _attn_device(ctx, q, k, v, bf16)


def _attn_device(ctx, q, k, v, bf16):
    """Device copies in the kernel layouts: rows padded to the kernel's tile
    multiple; bf16 V^T with the key order of the MFMA accumulator."""
    torch_cuda()
    heads, n, hd = q.shape
    npad = ctx.attn_pad(n)
    def pad(x):
        out = np.zeros((heads, npad, hd), np.float32)
        out[:, :n] = x
        return out
    qd, kd = ctx.to_device(pad(q)), ctx.to_device(pad(k))
    vp = pad(v)
    if bf16:
        # V^T layout of the bf16 kernel: key j stored at column j with bits 2 and 3 swapped
        j = np.arange(npad)
        pos = (j & ~12) | ((j & 4) << 1) | ((j & 8) >> 1)
        vt = np.zeros((heads, hd, npad), np.float32)
        vt[:, :, pos] = vp.transpose(0, 2, 1)
        vd = ctx.to_device(vt)
    else:
        vd = ctx.to_device(vp)
    return qd, kd, vd


def _heads_cfg(head_dim, heads):
    """A bf16 model descriptor with the given head count (only the attention shape matters)."""
    if heads is None:
        return small_cfg("bf16", head_dim=head_dim)
    return small_cfg("bf16", head_dim=head_dim, hidden=heads * head_dim, heads=heads)


# (head_dim, n, heads): heads None = the small model's (4 at hd 64, 2 at hd 128);
# head counts that are multiples of 8 take the per-XCD head order every real
# workload runs; n = 300 and 560 give 5 and 9 key tiles of 64
@pytest.mark.parametrize("head_dim,n,heads", [
    (64, 256, None), (64, 700, None), (64, 61, None), (64, 100, None), (64, 150, None), (64, 449, None),
    (64, 300, None), (64, 560, None), (64, 560, 16), (64, 1111, 24),
    (128, 512, None), (128, 1000, None), (128, 129, None), (128, 320, None), (128, 1111, None), (128, 61, None),
    (128, 100, None), (128, 150, None), (128, 256, None), (128, 1111, 8), (128, 600, 24)])
def test_attention_bf16_matches_oracle(head_dim, n, heads):
    torch = torch_cuda()
    cfg = _heads_cfg(head_dim, heads)
    ctx = context(cfg, weights=False)
    heads = cfg.heads
    (q, k, v), (qd, kd, vd) = _attn_inputs(ctx, heads, head_dim, n, seed=n, bf16=True)
    ldo = heads * head_dim + 32          # strided output rows
    out = torch.zeros((n, ldo), dtype=torch.bfloat16, device="cuda")
    ctx.attention(qd, kd, vd, n, out, ldo)
    got = out.float().cpu().numpy()
    ref = dit.attention(q, k, v).transpose(1, 0, 2).reshape(n, heads * head_dim)
    err = rel_l2(got[:, : heads * head_dim], ref)
    # per row and head
    rerr = row_rel_l2(got[:, : heads * head_dim].reshape(n, heads, head_dim), ref.reshape(n, heads, head_dim))
    print(f"hd {head_dim} n {n} heads {heads}: rel_l2 {err:.2e}, worst row {rerr:.2e}")
    assert err <= 1e-2, err
    assert rerr <= ROW_TOL_ATTN_BF16, rerr
    assert np.all(got[:, heads * head_dim:] == 0)      # nothing written past the heads


@pytest.mark.parametrize("head_dim", [64, 128])
def test_attention_bf16_score_jumps(head_dim):
    """Keys whose scores exceed every earlier key's by about 70 and then 140
    log2 units: the bf16 kernel must move its reference max twice mid-row (its
    P bound is 2^64 per lane sum), and a ragged last tile adds 14 more units."""
    torch = torch_cuda()
    cfg = small_cfg("bf16", head_dim=head_dim)
    ctx = context(cfg, weights=False)
    heads, n = cfg.heads, 700
    rng = _rng(4242 + head_dim)
    u = rng.standard_normal((heads, 1, head_dim))
    q = u + 0.1 * rng.standard_normal((heads, n, head_dim))
    k = rng.standard_normal((heads, n, head_dim))
    # log2-unit score of key c*u against q ~ u: c |u|^2 log2(e) / sqrt(hd) ~ 70 c / c1
    c1 = 70.0 * math.sqrt(head_dim) / (head_dim * math.log2(math.e))
    for lo, hi, c in ((192, 448, c1), (448, 640, 2 * c1), (640, n, 2.2 * c1)):
        k[:, lo:hi] = c * u + 0.1 * rng.standard_normal((heads, hi - lo, head_dim))
    v = rng.standard_normal((heads, n, head_dim))
    q, k, v = (synth.round_bf16(x).astype(np.float64) for x in (q, k, v))
    qd, kd, vd = _attn_device(ctx, q, k, v, bf16=True)
    ldo = heads * head_dim
    out = torch.zeros((n, ldo), dtype=torch.bfloat16, device="cuda")
    ctx.attention(qd, kd, vd, n, out, ldo)
    got = out.float().cpu().numpy()
    ref = dit.attention(q, k, v).transpose(1, 0, 2).reshape(n, ldo)
    err = rel_l2(got, ref)
    print("head_dim", head_dim, "rel_l2", err)
    assert np.all(np.isfinite(got)) and err <= 1e-2, err


def test_attention_rejects_bad_output_layout():
    """ldo below heads*hd (rows would overlap and the last row overrun its
    buffer) and a bf16 output stride that breaks the 8-byte column groups."""
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    cfg = small_cfg("bf16", head_dim=128)
    ctx = context(cfg, weights=False)
    heads, hd, n = cfg.heads, 128, 100
    _, (qd, kd, vd) = _attn_inputs(ctx, heads, hd, n, seed=5, bf16=True)
    out = torch.zeros((n, heads * hd + 8), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(wdc.WdcError):
        ctx.attention(qd, kd, vd, n, out, heads * hd - 4)
    with pytest.raises(wdc.WdcError):
        ctx.attention(qd, kd, vd, n, out, heads * hd + 2)
    ctx.attention(qd, kd, vd, n, out, heads * hd + 8)       # a valid stride still works
    assert torch.isfinite(out.float()).all()


@pytest.mark.parametrize("head_dim,n", [(64, 256), (64, 77), (128, 100)])
def test_attention_f32_matches_oracle(head_dim, n):
    torch = torch_cuda()
    cfg = small_cfg("f32", head_dim=head_dim)
    ctx = context(cfg, weights=False)
    (q, k, v), (qd, kd, vd) = _attn_inputs(ctx, cfg.heads, head_dim, n, seed=n + 1, bf16=False)
    ldo = cfg.heads * head_dim
    out = torch.zeros((n, ldo), dtype=torch.float32, device="cuda")
    ctx.attention(qd, kd, vd, n, out, ldo)
    ref = dit.attention(q, k, v).transpose(1, 0, 2).reshape(n, ldo)
    assert rel_l2(out.cpu().numpy(), ref) <= TOL_F32


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_cond_embed_matches_oracle(dtype):
    torch = torch_cuda()
    cfg = small_cfg(dtype)
    ctx = context(cfg)
    W = synth.gen_weights(cfg)
    inp = synth.gen_inputs(cfg)
    for t in (1.0, 0.55, 0.0):
        got = ctx.cond_embed(t, ctx.to_device(inp["cond"]), ctx.to_device(inp["cam"])).cpu().numpy()
        ref = dit.cond_embedding(W, cfg, t, inp["cond"], inp["cam"])
        assert rel_l2(got, ref) <= TOL_F32     # same (bf16-valued) weights, float32 accumulation
