"""Pins for the oracle denoiser (oracle/dit.py), CPU only.

Each check is tied to something outside the oracle's own code: brute force
loops, closed forms, invariants, or an independent formulation built from
library routines (torch CPU functional ops in float64).
"""
import math
from dataclasses import replace

import numpy as np
import pytest
import torch
import torch.nn.functional as tF

import synth
from oracle import dit

RNG = np.random.default_rng(1234)


def small_cfg(**kw):
    base = dict(name="unit", dtype="f32", hidden=64, heads=2, head_dim=32, n_seq=1, n_dual=1, n_single=1,
                cond_dim=8, cam_dim=6, text_tokens=3, text_dim=10, latent=(16, 2, 4, 6),
                patch=(1, 2, 2), rope=(8, 12, 12), steps=4, seed=7)
    base.update(kw)
    return synth.ModelConfig(**base)


# --------------------------------------------------------------------------- elementary ops

def test_layer_norm_matches_library_and_moments():
    x = RNG.standard_normal((5, 48)) * 3 + 1
    y = dit.layer_norm(x)
    ref = tF.layer_norm(torch.tensor(x), (48,), eps=1e-6).numpy()
    np.testing.assert_allclose(y, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-12)
    np.testing.assert_allclose(y.var(-1), 1, atol=1e-5)


def test_rms_norm_unit_rms_and_library():
    x = RNG.standard_normal((4, 32)) * 5
    y = dit.rms_norm(x)
    np.testing.assert_allclose(np.sqrt((y * y).mean(-1)), 1, atol=1e-6)
    ref = tF.rms_norm(torch.tensor(x), (32,), eps=1e-6).numpy()
    np.testing.assert_allclose(y, ref, atol=1e-12)


def test_gelu_tanh_matches_library():
    x = np.linspace(-8, 8, 1001)
    ref = tF.gelu(torch.tensor(x), approximate="tanh").numpy()
    np.testing.assert_allclose(dit.gelu_tanh(x), ref, atol=1e-14)
    assert dit.gelu_tanh(np.array([0.0]))[0] == 0.0


def test_silu_closed_form():
    x = np.linspace(-10, 10, 101)
    np.testing.assert_allclose(dit.silu(x), tF.silu(torch.tensor(x)).numpy(), atol=1e-14)


def test_timestep_features_closed_form():
    f0 = dit.timestep_features(0.0)
    np.testing.assert_array_equal(f0[:128], 1.0)
    np.testing.assert_array_equal(f0[128:], 0.0)
    t = 0.37
    f = dit.timestep_features(t)
    # j = 0 has frequency 1; j = 64 has frequency 1e4^(-1/2) = 0.01
    assert f[0] == pytest.approx(math.cos(370.0), abs=1e-12)
    assert f[128] == pytest.approx(math.sin(370.0), abs=1e-12)
    assert f[64] == pytest.approx(math.cos(3.7), abs=1e-12)
    assert f[192] == pytest.approx(math.sin(3.7), abs=1e-12)


def test_linear_matches_library():
    W = {"l.w": RNG.standard_normal((7, 5)), "l.b": RNG.standard_normal(7)}
    x = RNG.standard_normal((3, 5))
    ref = tF.linear(torch.tensor(x), torch.tensor(W["l.w"]), torch.tensor(W["l.b"])).numpy()
    np.testing.assert_allclose(dit.linear(W, "l", x), ref, atol=1e-13)
    np.testing.assert_allclose(dit.linear_rows(W, "l", x, 2, 5), ref[:, 2:5], atol=1e-13)


# --------------------------------------------------------------------------- attention

def brute_attention(q, k, v):
    hh, nq, hd = q.shape
    nk = k.shape[1]
    out = np.zeros((hh, nq, v.shape[2]))
    for h in range(hh):
        for i in range(nq):
            s = [sum(q[h, i, d] * k[h, j, d] for d in range(hd)) / math.sqrt(hd) for j in range(nk)]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = sum(e)
            for j in range(nk):
                for d in range(v.shape[2]):
                    out[h, i, d] += e[j] / z * v[h, j, d]
    return out


def test_attention_brute_force():
    q, k, v = (RNG.standard_normal((2, n, 8)) for n in (5, 7, 7))
    np.testing.assert_allclose(dit.attention(q, k, v), brute_attention(q, k, v), atol=1e-12)


def test_attention_chunking_does_not_change_result():
    q, k, v = (RNG.standard_normal((3, 37, 16)) for _ in range(3))
    np.testing.assert_allclose(dit.attention(q, k, v, chunk=5), dit.attention(q, k, v, chunk=1024), atol=1e-13)


def test_attention_library_sdpa():
    q, k, v = (RNG.standard_normal((4, 33, 64)) for _ in range(3))
    ref = tF.scaled_dot_product_attention(torch.tensor(q), torch.tensor(k), torch.tensor(v)).numpy()
    np.testing.assert_allclose(dit.attention(q, k, v), ref, atol=1e-12)


def test_attention_special_cases():
    # identical keys: every weight is 1/N, output = mean of V
    q = RNG.standard_normal((1, 4, 8))
    k = np.repeat(RNG.standard_normal((1, 1, 8)), 9, axis=1)
    v = RNG.standard_normal((1, 9, 8))
    np.testing.assert_allclose(dit.attention(q, k, v), np.broadcast_to(v.mean(1, keepdims=True), (1, 4, 8)), atol=1e-13)
    # one dominant score selects that row of V
    k2 = np.zeros((1, 6, 8)); k2[0, 3, 0] = 1e3
    q2 = np.zeros((1, 1, 8)); q2[0, 0, 0] = 1.0
    v2 = RNG.standard_normal((1, 6, 8))
    np.testing.assert_allclose(dit.attention(q2, k2, v2)[0, 0], v2[0, 3], atol=1e-12)
    # one vector added to every key adds q.c to a whole row of scores: no change (softmax shift)
    q3, k3, v3 = (RNG.standard_normal((1, 5, 8)) for _ in range(3))
    k3b = k3 + RNG.standard_normal((1, 1, 8))
    np.testing.assert_allclose(dit.attention(q3, k3b, v3), dit.attention(q3, k3, v3), atol=1e-13)


# --------------------------------------------------------------------------- RoPE

def test_rope_matches_complex_rotation():
    grid, dims = (2, 3, 4), (4, 6, 6)
    ang = dit.rope_angles(grid, dims)
    x = RNG.standard_normal((2, 24, 16))
    y = dit.apply_rope(x, ang)
    # independent formulation: pairs as complex numbers times e^{i*angle}
    pos = [(f, h, w) for f in range(2) for h in range(3) for w in range(4)]
    for n, (f, h, w) in enumerate(pos):
        th = []
        for p_, d in zip((f, h, w), dims):
            th += [p_ * 10000.0 ** (-2.0 * j / d) for j in range(d // 2)]
        zc = (x[:, n, 0::2] + 1j * x[:, n, 1::2]) * np.exp(1j * np.array(th))
        np.testing.assert_allclose(y[:, n, 0::2], zc.real, atol=1e-12)
        np.testing.assert_allclose(y[:, n, 1::2], zc.imag, atol=1e-12)


def test_rope_invariants():
    grid, dims = (3, 4, 5), (4, 6, 6)
    ang = dit.rope_angles(grid, dims)
    x = RNG.standard_normal((1, 60, 16))
    y = dit.apply_rope(x, ang)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)
    np.testing.assert_array_equal(y[:, 0], x[:, 0])          # position (0,0,0) is the identity
    # <R_m q, R_n k> depends only on m - n (per axis): shift both tokens by one frame
    q, k = RNG.standard_normal(16), RNG.standard_normal(16)
    pos = dit.token_positions(grid)
    idx = {tuple(p): i for i, p in enumerate(pos)}
    def dot(a, b):
        ra = dit.apply_rope(q[None], ang[[idx[a]]])[0]
        rb = dit.apply_rope(k[None], ang[[idx[b]]])[0]
        return ra @ rb
    assert dot((0, 1, 2), (1, 3, 0)) == pytest.approx(dot((1, 1, 2), (2, 3, 0)), abs=1e-12)
    assert dot((0, 0, 1), (0, 2, 4)) == pytest.approx(dot((0, 1, 0), (0, 3, 3)), abs=1e-12)


# --------------------------------------------------------------------------- patches

def test_patchify_layout_and_roundtrip():
    z = RNG.standard_normal((16, 2, 4, 6))
    tok = dit.patchify(z, (1, 2, 2))
    assert tok.shape == (2 * 2 * 3, 64)
    # token (f=1, h'=1, w'=2) is index (1*2 + 1)*3 + 2 = 11; feature (c=5, i=1, j=0) = 5*4 + 2
    assert tok[11, 5 * 4 + 2] == z[5, 1, 3, 4]
    np.testing.assert_array_equal(dit.unpatchify(tok, z.shape, (1, 2, 2)), z)
    z2 = RNG.standard_normal((16, 4, 4, 4))
    tok2 = dit.patchify(z2, (2, 2, 2))
    assert tok2[0, 3 * 8 + 1 * 4 + 1 * 2 + 0] == z2[3, 1, 1, 0]
    np.testing.assert_array_equal(dit.unpatchify(tok2, z2.shape, (2, 2, 2)), z2)


# --------------------------------------------------------------------------- blocks vs torch

def T(a):
    return torch.tensor(np.asarray(a, dtype=np.float64))


def torch_rope(t, ang, n_video):
    """t: [H, N, hd]; rotate video rows with complex multiplication."""
    out = t.clone()
    tv = t[:, :n_video].reshape(t.shape[0], n_video, -1, 2)
    zc = torch.view_as_complex(tv.contiguous())
    rot = torch.polar(torch.ones_like(T(ang)), T(ang))
    out[:, :n_video] = torch.view_as_real(zc * rot).reshape(t.shape[0], n_video, -1)
    return out


def torch_attn(cfg, q, k, v, ang):
    def heads(x):
        return x.reshape(x.shape[0], cfg.heads, cfg.head_dim).transpose(0, 1)
    q, k, v = heads(q), heads(k), heads(v)
    q = tF.rms_norm(q, (cfg.head_dim,), eps=1e-6)
    k = tF.rms_norm(k, (cfg.head_dim,), eps=1e-6)
    q, k = torch_rope(q, ang, cfg.n_video), torch_rope(k, ang, cfg.n_video)
    o = tF.scaled_dot_product_attention(q, k, v)
    return o.transpose(0, 1).reshape(-1, cfg.hidden)


def torch_block(W, cfg, b, x, c):
    """Independent composition of a block from torch functional ops."""
    d = cfg.hidden
    x, c = T(x), T(c)
    lin = lambda n, y: tF.linear(y, T(W[n + ".w"]), T(W[n + ".b"]))
    ln = lambda y: tF.layer_norm(y, (d,), eps=1e-6)
    ang = dit.rope_angles(cfg.grid, cfg.rope)
    kind, pre = dit.block_kind(cfg, b), dit.block_prefix(cfg, b)
    sc = tF.silu(c)
    if kind == "seq":
        m = lin(pre + ".ada", sc).chunk(6)
        h = ln(x) * (1 + m[1]) + m[0]
        q, k, v = lin(pre + ".qkv", h).chunk(3, dim=-1)
        x = x + m[2] * lin(pre + ".out", torch_attn(cfg, q, k, v, ang))
        h = ln(x) * (1 + m[4]) + m[3]
        return (x + m[5] * lin(pre + ".fc2", tF.gelu(lin(pre + ".fc1", h), approximate="tanh"))).numpy()
    if kind == "dual":
        nv = cfg.n_video
        mv, mt = lin(pre + ".vid.ada", sc).chunk(6), lin(pre + ".txt.ada", sc).chunk(6)
        xv, xt = x[:nv], x[nv:]
        qv, kv, vv = lin(pre + ".vid.qkv", ln(xv) * (1 + mv[1]) + mv[0]).chunk(3, dim=-1)
        qt, kt, vt = lin(pre + ".txt.qkv", ln(xt) * (1 + mt[1]) + mt[0]).chunk(3, dim=-1)
        o = torch_attn(cfg, torch.cat([qv, qt]), torch.cat([kv, kt]), torch.cat([vv, vt]), ang)
        outs = []
        for s, xs, ms, os_ in (("vid", xv, mv, o[:nv]), ("txt", xt, mt, o[nv:])):
            xs = xs + ms[2] * lin(f"{pre}.{s}.out", os_)
            h = ln(xs) * (1 + ms[4]) + ms[3]
            outs.append(xs + ms[5] * lin(f"{pre}.{s}.fc2", tF.gelu(lin(f"{pre}.{s}.fc1", h), approximate="tanh")))
        return torch.cat(outs).numpy()
    m = lin(pre + ".ada", sc).chunk(3)
    h = ln(x) * (1 + m[1]) + m[0]
    y = lin(pre + ".lin1", h)
    q, k, v, mm = y[:, :d], y[:, d:2 * d], y[:, 2 * d:3 * d], y[:, 3 * d:]
    cat = torch.cat([torch_attn(cfg, q, k, v, ang), tF.gelu(mm, approximate="tanh")], dim=1)
    return (x + m[2] * lin(pre + ".lin2", cat)).numpy()


@pytest.mark.parametrize("block", [0, 1, 2])
def test_blocks_match_torch_composition(block):
    cfg = small_cfg()
    W = {k: v.astype(np.float64) * 5 for k, v in synth.gen_weights(cfg).items()}   # larger weights: visible updates
    x = RNG.standard_normal((cfg.n_tokens, cfg.hidden))
    c = RNG.standard_normal(cfg.hidden)
    got = dit.block_forward(W, cfg, block, x, c)
    ref = torch_block(W, cfg, block, x, c)
    assert np.abs(got - x).max() > 1e-2          # the block does something
    np.testing.assert_allclose(got, ref, atol=1e-11)


@pytest.mark.parametrize("block", [0, 1, 2])
def test_block_rows_subset_equals_full(block):
    cfg = small_cfg()
    W = synth.gen_weights(cfg)
    x = RNG.standard_normal((cfg.n_tokens, cfg.hidden))
    c = RNG.standard_normal(cfg.hidden)
    full = dit.block_forward(W, cfg, block, x, c)
    rows = np.array([0, 5, cfg.n_video - 1, cfg.n_video, cfg.n_tokens - 1])
    np.testing.assert_allclose(dit.block_forward(W, cfg, block, x, c, rows=rows), full[rows], atol=1e-13)


@pytest.mark.parametrize("block", [0, 1, 2])
def test_zero_gate_block_is_identity(block):
    """adaLN with zero modulation weights and biases gives gates of 0: the block is the identity."""
    cfg = small_cfg()
    W = dict(synth.gen_weights(cfg))
    for k in list(W):
        if ".ada." in k:
            W[k] = np.zeros_like(W[k])
    x = RNG.standard_normal((cfg.n_tokens, cfg.hidden))
    np.testing.assert_array_equal(dit.block_forward(W, cfg, block, x, RNG.standard_normal(cfg.hidden)), x)


def test_attention_invariant_to_global_position_shift():
    """With RoPE, shifting every video position by the same offset leaves scores unchanged."""
    cfg = small_cfg()
    ang = dit.rope_angles(cfg.grid, cfg.rope)
    # angles for positions shifted by +1 along every axis
    pos = dit.token_positions(cfg.grid).astype(float) + 1.0
    parts = []
    for a, d in enumerate(cfg.rope):
        j = np.arange(d // 2)
        parts.append(np.outer(pos[:, a], 10000.0 ** (-2.0 * j / d)))
    ang2 = np.concatenate(parts, 1)
    q, k, v = (RNG.standard_normal((2, cfg.n_video, cfg.head_dim)) for _ in range(3))
    a1 = dit.attention(dit.apply_rope(q, ang), dit.apply_rope(k, ang), v)
    a2 = dit.attention(dit.apply_rope(q, ang2), dit.apply_rope(k, ang2), v)
    np.testing.assert_allclose(a1, a2, atol=1e-12)


def test_forward_final_layer_and_conditioning():
    cfg = small_cfg()
    W = synth.gen_weights(cfg)
    inp = synth.gen_inputs(cfg)
    v = dit.dit_forward(W, cfg, inp["z_T"], 0.5, inp["cond"], inp["text"], inp["cam"])
    assert v.shape == cfg.latent and np.all(np.isfinite(v))
    # conditioning: timestep MLP plus linear condition and camera terms, by torch
    c = tF.linear(tF.silu(tF.linear(T(dit.timestep_features(0.5)), T(W["t_embed.fc1.w"]), T(W["t_embed.fc1.b"]))),
                  T(W["t_embed.fc2.w"]), T(W["t_embed.fc2.b"]))
    c = c + tF.linear(T(inp["cond"]), T(W["cond_embed.w"]), T(W["cond_embed.b"]))
    c = c + tF.linear(T(inp["cam"]), T(W["cam_embed.w"]), T(W["cam_embed.b"]))
    np.testing.assert_allclose(dit.cond_embedding(W, cfg, 0.5, inp["cond"], inp["cam"]), c.numpy(), atol=1e-13)
    # the output head only reads video tokens: changing text-token rows of the stream leaves v alone
    x = dit.embed_tokens(W, cfg, inp["z_T"], inp["text"])
    cemb = c.numpy()
    v1 = dit.final_layer(W, cfg, x[: cfg.n_video], cemb)
    x[cfg.n_video:] += 100
    np.testing.assert_array_equal(dit.final_layer(W, cfg, x[: cfg.n_video], cemb), v1)


# --------------------------------------------------------------------------- whole F_theta vs torch

def torch_forward(W, cfg, z, t, cond=None, text=None, cam=None):
    """Independent composition of F_theta from torch library ops: the patch
    embedding as a strided 3D convolution, the blocks of ``torch_block``, the
    output head by torch LayerNorm / SiLU / linear and unpatchify by einops."""
    import einops
    d, half = cfg.hidden, 128
    lin = lambda n, y: tF.linear(y, T(W[n + ".w"]), T(W[n + ".b"]))
    freqs = torch.exp(-math.log(10000.0) * torch.arange(half, dtype=torch.float64) / half)
    ang = 1000.0 * t * freqs
    c = lin("t_embed.fc2", tF.silu(lin("t_embed.fc1", torch.cat([torch.cos(ang), torch.sin(ang)]))))
    if cfg.cond_dim:
        c = c + lin("cond_embed", T(cond))
    if cfg.cam_dim:
        c = c + lin("cam_embed", T(cam))
    ch = cfg.latent[0]
    kern = T(W["patch_embed.w"]).reshape(d, ch, *cfg.patch)
    x = tF.conv3d(T(z)[None], kern, T(W["patch_embed.b"]), stride=tuple(cfg.patch))[0]   # [D, F', H', W']
    x = x.reshape(d, -1).T
    if cfg.text_tokens:
        x = torch.cat([x, lin("text_proj", T(text))])
    for b in range(cfg.n_blocks):
        x = T(torch_block(W, cfg, b, x.numpy(), c.numpy()))
    shift, scale = lin("final.ada", tF.silu(c)).chunk(2)
    h = tF.layer_norm(x[: cfg.n_video], (d,), eps=1e-6) * (1 + scale) + shift
    out = lin("final.lin", h)
    fp, hp, wp = cfg.grid
    pt, ph, pw = cfg.patch
    return einops.rearrange(out.numpy(), "(f h w) (c a i j) -> c (f a) (h i) (w j)", f=fp, h=hp, w=wp,
                            c=ch, a=pt, i=ph, j=pw)


def _forward_case(**kw):
    cfg = small_cfg(**kw)
    W = {k: v.astype(np.float64) * 5 for k, v in synth.gen_weights(cfg).items()}    # visible modulation
    inp = synth.gen_inputs(cfg)
    return cfg, W, inp


@pytest.mark.parametrize("patch,t", [((1, 2, 2), 0.62), ((2, 2, 2), 0.25)])
def test_dit_forward_matches_torch_composition(patch, t):
    """The whole F_theta (conditioning, patch embedding, all three block kinds
    over the joint sequence, the output head and unpatchify) against the torch
    composition."""
    cfg, W, inp = _forward_case(patch=patch)
    got = dit.dit_forward(W, cfg, inp["z_T"], t, inp["cond"], inp["text"], inp["cam"])
    ref = torch_forward(W, cfg, inp["z_T"], t, inp["cond"], inp["text"], inp["cam"])
    assert np.abs(ref).max() > 1e-2
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10 * np.abs(ref).max())


def _final_swapped(W, cfg, x_video, c_emb):
    scale, shift = np.split(dit.linear(W, "final.ada", dit.silu(c_emb)), 2)
    out = dit.linear(W, "final.lin", dit.modulate(dit.layer_norm(x_video), shift, scale))
    return dit.unpatchify(out, cfg.latent, cfg.patch)


def _final_no_silu(W, cfg, x_video, c_emb):
    shift, scale = np.split(dit.linear(W, "final.ada", c_emb), 2)
    out = dit.linear(W, "final.lin", dit.modulate(dit.layer_norm(x_video), shift, scale))
    return dit.unpatchify(out, cfg.latent, cfg.patch)


def _final_no_norm(W, cfg, x_video, c_emb):
    shift, scale = np.split(dit.linear(W, "final.ada", dit.silu(c_emb)), 2)
    out = dit.linear(W, "final.lin", dit.modulate(x_video, shift, scale))
    return dit.unpatchify(out, cfg.latent, cfg.patch)


@pytest.mark.parametrize("mistake", [_final_swapped, _final_no_silu, _final_no_norm])
def test_output_head_mistakes_are_caught(monkeypatch, mistake):
    """Plausible mistakes planted in the oracle's output head (shift and scale
    swapped, SiLU dropped, LayerNorm dropped) make it disagree with the torch
    composition, so the comparison above pins the head."""
    cfg, W, inp = _forward_case()
    ref = torch_forward(W, cfg, inp["z_T"], 0.62, inp["cond"], inp["text"], inp["cam"])
    monkeypatch.setattr(dit, "final_layer", mistake)
    bad = dit.dit_forward(W, cfg, inp["z_T"], 0.62, inp["cond"], inp["text"], inp["cam"])
    assert np.abs(bad - ref).max() > 1e-3 * np.abs(ref).max()


def test_output_head_matches_torch():
    """The output head alone: torch LayerNorm, SiLU and linear, then einops unpatchify."""
    import einops
    cfg, W, inp = _forward_case()
    x = RNG.standard_normal((cfg.n_video, cfg.hidden)) * 2 + 0.5
    c = RNG.standard_normal(cfg.hidden)
    shift, scale = tF.linear(tF.silu(T(c)), T(W["final.ada.w"]), T(W["final.ada.b"])).chunk(2)
    h = tF.layer_norm(T(x), (cfg.hidden,), eps=1e-6) * (1 + scale) + shift
    out = tF.linear(h, T(W["final.lin.w"]), T(W["final.lin.b"])).numpy()
    fp, hp, wp = cfg.grid
    ref = einops.rearrange(out, "(f h w) (c a i j) -> c (f a) (h i) (w j)", f=fp, h=hp, w=wp, c=16, a=1, i=2, j=2)
    np.testing.assert_allclose(dit.final_layer(W, cfg, x, c), ref, atol=1e-12 * np.abs(ref).max())


# --------------------------------------------------------------------------- whole-forward invariants

def _head_permuted(W, cfg, perm):
    """The weights with the attention heads relabelled by ``perm``: the q, k and v
    output rows of every projection move by whole heads, and the attention-output
    columns of every output projection follow. The model is unchanged."""
    d, hd = cfg.hidden, cfg.head_dim
    cols = np.concatenate([np.arange(p * hd, (p + 1) * hd) for p in perm])
    rows = np.concatenate([cols, d + cols, 2 * d + cols])
    V = dict(W)
    for name in W:
        if name.endswith((".qkv.w", ".qkv.b")):
            V[name] = W[name][rows]
        elif name.endswith(".lin1.w") or name.endswith(".lin1.b"):
            V[name] = np.concatenate([W[name][rows], W[name][3 * d:]])
        elif name.endswith(".out.w"):
            V[name] = W[name][:, cols]
        elif name.endswith(".lin2.w"):
            V[name] = np.concatenate([W[name][:, cols], W[name][:, d:]], axis=1)
    return V


def test_dit_forward_invariant_to_head_relabelling():
    """Per-head RMSNorm and RoPE act alike on every head and the joint attention
    is per head, so relabelling the heads consistently in every block (both
    streams of the dual block included) leaves F_theta unchanged; a mismatch
    between the head split and the head merge, or streams split differently,
    breaks it."""
    cfg = small_cfg(heads=4, head_dim=16, rope=(4, 6, 6))
    W = {k: v.astype(np.float64) * 5 for k, v in synth.gen_weights(cfg).items()}
    inp = synth.gen_inputs(cfg)
    args = (inp["z_T"], 0.4, inp["cond"], inp["text"], inp["cam"])
    ref = dit.dit_forward(W, cfg, *args)
    got = dit.dit_forward(_head_permuted(W, cfg, [2, 0, 3, 1]), cfg, *args)
    assert np.abs(ref).max() > 1e-2
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10 * np.abs(ref).max())
    # a relabelling of the q/k rows alone (v and the output columns left) is a different model
    bad = dict(W)
    for name in W:
        if name.endswith((".qkv.w", ".qkv.b")):
            d, hd = cfg.hidden, cfg.head_dim
            cols = np.concatenate([np.arange(p * hd, (p + 1) * hd) for p in [2, 0, 3, 1]])
            bad[name] = W[name][np.concatenate([cols, d + cols, 2 * d + np.arange(d)])]
    assert np.abs(dit.dit_forward(bad, cfg, *args) - ref).max() > 1e-3 * np.abs(ref).max()


def test_dit_forward_invariant_to_text_token_order():
    """Text tokens carry no position (RoPE rotates the video rows only) and every
    video query attends over the joint set of keys, so reordering the text
    tokens leaves the velocity unchanged; giving text rows a position or
    attending over the video rows alone would break it (the second is checked:
    dropping the text changes the velocity)."""
    cfg = small_cfg(text_tokens=5)
    W = {k: v.astype(np.float64) * 5 for k, v in synth.gen_weights(cfg).items()}
    inp = synth.gen_inputs(cfg)
    text = inp["text"]
    ref = dit.dit_forward(W, cfg, inp["z_T"], 0.7, inp["cond"], text, inp["cam"])
    got = dit.dit_forward(W, cfg, inp["z_T"], 0.7, inp["cond"], text[[3, 0, 4, 2, 1]], inp["cam"])
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10 * np.abs(ref).max())
    other = dit.dit_forward(W, cfg, inp["z_T"], 0.7, inp["cond"], 2.0 * text, inp["cam"])
    assert np.abs(other - ref).max() > 1e-3 * np.abs(ref).max()


def test_dit_forward_with_zero_gates_is_the_output_head_on_the_embedding():
    """With every block's residual gates zero (their adaLN rows and biases zeroed,
    shift and scale left as they are) each block returns its input, so F_theta
    reduces to the output head applied to the patch embedding; a block that
    added its branch ungated, or replaced the stream by its modulated input,
    would not."""
    cfg = small_cfg()
    W = {k: v.astype(np.float64) * 5 for k, v in synth.gen_weights(cfg).items()}
    d = cfg.hidden
    for name in list(W):
        if name.endswith((".ada.w", ".ada.b")) and not name.startswith("final"):
            gates = [2] if name.startswith("single") else [2, 5]
            W[name] = W[name].copy()
            for g in gates:
                W[name][g * d:(g + 1) * d] = 0.0
    inp = synth.gen_inputs(cfg)
    args = (inp["z_T"], 0.55, inp["cond"], inp["text"], inp["cam"])
    got = dit.dit_forward(W, cfg, *args)
    c_emb = dit.cond_embedding(W, cfg, 0.55, inp["cond"], inp["cam"])
    tokens = dit.patchify(np.asarray(inp["z_T"], np.float64), cfg.patch) @ W["patch_embed.w"].T + W["patch_embed.b"]
    ref = dit.final_layer(W, cfg, tokens, c_emb)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * np.abs(ref).max())


def _merge_interleaved(x):
    h, n, hd = x.shape
    return x.transpose(1, 2, 0).reshape(n, h * hd)


def _rope_on_text(cfg, n_rows):
    idx = np.arange(n_rows)
    return np.where(idx < cfg.n_video, idx, idx % cfg.n_video)


_single_block = dit.single_block


def _single_stream_replaced(W, cfg, pre, x, c_emb, rows=None):
    sh, sc, _ = np.split(dit.linear(W, pre + ".ada", dit.silu(c_emb)), 3)
    return _single_block(W, cfg, pre, x, c_emb, rows) + dit.modulate(dit.layer_norm(x), sh, sc) - x


@pytest.mark.parametrize("target,mistake,test", [
    ("_merge", _merge_interleaved, test_dit_forward_invariant_to_head_relabelling),
    ("_rope_index", _rope_on_text, test_dit_forward_invariant_to_text_token_order),
    ("single_block", _single_stream_replaced, test_dit_forward_with_zero_gates_is_the_output_head_on_the_embedding),
])
def test_whole_forward_invariants_catch_planted_mistakes(monkeypatch, target, mistake, test):
    """Each whole-forward invariant fails on the oracle with a plausible mistake
    planted: heads merged in an interleaved order after a contiguous split,
    text rows rotated as if they had video positions, a single-stream block
    whose stream is replaced by its modulated input."""
    monkeypatch.setattr(dit, target, mistake)
    with pytest.raises(AssertionError):
        test()
