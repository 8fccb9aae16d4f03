"""Oracle denoiser F_theta: a synthetic video diffusion transformer, float64.

The paper treats the denoiser F_theta of Eq. (1) as a given large video
transformer (Sec. 1, Sec. 4.1) and never specifies it. This module defines
the stand-in used throughout: a DiT with adaLN modulation, per-head
QK-RMSNorm, 3D rotary position embedding on video tokens and a GELU-tanh MLP,
in three block kinds:

* sequential block: x += g1*Attn(mod(LN x)); x += g2*MLP(mod(LN x)), shared
  weights over the joint [video; text] sequence;
* dual-stream block: per-stream weights and modulation for video and text
  tokens, one attention over the joint sequence;
* single-stream block: one linear producing [q, k, v, mlp-in], one linear
  mapping [attn-out, GELU(mlp-in)] back, gated residual.

Everything is evaluated straight from its definition (row-chunked attention
is only a memory bound on the same arithmetic). ``rows`` arguments evaluate a
block's output at selected token rows; keys and values still come from every
token, which is exact because all other operations act token by token.
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Sequence

import numpy as np

LN_EPS = 1e-6
RMS_EPS = 1e-6
ROPE_BASE = 10000.0


def f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# elementary operations
# ---------------------------------------------------------------------------

def layer_norm(x: np.ndarray, eps: float = LN_EPS) -> np.ndarray:
    """LayerNorm over the last axis without affine parameters (biased variance)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def rms_norm(x: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps)


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def modulate(x: np.ndarray, shift: np.ndarray, scale: np.ndarray) -> np.ndarray:
    return x * (1.0 + scale) + shift


def linear(W: Dict[str, np.ndarray], name: str, x: np.ndarray) -> np.ndarray:
    """x @ weight.T + bias with weight stored [out, in]."""
    return x @ f64(W[name + ".w"]).T + f64(W[name + ".b"])


def linear_rows(W: Dict[str, np.ndarray], name: str, x: np.ndarray, r0: int, r1: int) -> np.ndarray:
    """Output features [r0, r1) of a linear layer."""
    return x @ f64(W[name + ".w"][r0:r1]).T + f64(W[name + ".b"][r0:r1])


def timestep_features(t: float, dim: int = 256) -> np.ndarray:
    """Sinusoidal features of 1000*t: [cos(1000 t f_j), sin(1000 t f_j)], f_j = 1e4^(-j/(dim/2))."""
    half = dim // 2
    freqs = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    arg = 1000.0 * float(t) * freqs
    return np.concatenate([np.cos(arg), np.sin(arg)])


# ---------------------------------------------------------------------------
# positions
# ---------------------------------------------------------------------------

def token_positions(grid: Sequence[int]) -> np.ndarray:
    """[N_v, 3] integer (f, h, w) of video token n = (f*H' + h)*W' + w."""
    fp, hp, wp = grid
    f, h, w = np.meshgrid(np.arange(fp), np.arange(hp), np.arange(wp), indexing="ij")
    return np.stack([f.ravel(), h.ravel(), w.ravel()], axis=1)


def rope_angles(grid: Sequence[int], axis_dims: Sequence[int], base: float = ROPE_BASE) -> np.ndarray:
    """[N_v, hd/2] rotation angles. Axis a owns a contiguous section of
    ``axis_dims[a]`` head dimensions split into interleaved pairs (2j, 2j+1);
    pair j of that section turns by pos_a * base^(-2j/d_a)."""
    pos = token_positions(grid).astype(np.float64)
    parts = []
    for a, d in enumerate(axis_dims):
        j = np.arange(d // 2, dtype=np.float64)
        parts.append(np.outer(pos[:, a], base ** (-2.0 * j / d)))
    return np.concatenate(parts, axis=1)


def apply_rope(x: np.ndarray, ang: np.ndarray) -> np.ndarray:
    """Rotate pairs (x[2i], x[2i+1]) by ang[..., i]. x: [..., n, hd], ang: [n, hd/2]."""
    x0, x1 = x[..., 0::2], x[..., 1::2]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    out[..., 0::2] = x0 * c - x1 * s
    out[..., 1::2] = x0 * s + x1 * c
    return out


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, chunk: int = 1024) -> np.ndarray:
    """softmax(q k^T / sqrt(hd)) v per head, non-causal. q: [H, Nq, hd]; k, v: [H, Nk, hd]."""
    hh, nq, hd = q.shape
    scale = 1.0 / math.sqrt(hd)
    out = np.empty((hh, nq, v.shape[-1]), dtype=np.float64)
    for h in range(hh):
        for r0 in range(0, nq, chunk):
            s = (q[h, r0:r0 + chunk] @ k[h].T) * scale
            s = s - s.max(axis=-1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=-1, keepdims=True)
            out[h, r0:r0 + chunk] = p @ v[h]
    return out


def _heads(x: np.ndarray, heads: int) -> np.ndarray:
    n, d = x.shape
    return x.reshape(n, heads, d // heads).transpose(1, 0, 2)


def _merge(x: np.ndarray) -> np.ndarray:
    h, n, hd = x.shape
    return x.transpose(1, 0, 2).reshape(n, h * hd)


def _prep_qk(x: np.ndarray, cfg, rope_rows: Optional[np.ndarray], ang: np.ndarray) -> np.ndarray:
    """[n, D] -> [H, n, hd] with per-head RMSNorm and RoPE on the video rows.
    ``rope_rows``: for each row, its video token index or -1 for text rows."""
    t = _heads(x, cfg.heads)
    if cfg.qk_norm:
        t = rms_norm(t)
    if ang is not None:
        vid = rope_rows >= 0
        if vid.any():
            t = t.copy()
            t[:, vid] = apply_rope(t[:, vid], ang[rope_rows[vid]])
    return t


def _rope_index(cfg, n_rows: int) -> np.ndarray:
    idx = np.arange(n_rows)
    return np.where(idx < cfg.n_video, idx, -1)


def _angles(cfg):
    return rope_angles(cfg.grid, cfg.rope) if sum(cfg.rope) else None


# ---------------------------------------------------------------------------
# conditioning, patch embedding and output head
# ---------------------------------------------------------------------------

def cond_embedding(W, cfg, t: float, cond=None, cam=None) -> np.ndarray:
    """c_emb = MLP(sinusoid(t)) + Linear(cond) + Linear(cam) (the last two when present)."""
    e = linear(W, "t_embed.fc2", silu(linear(W, "t_embed.fc1", timestep_features(t))))
    if cfg.cond_dim:
        e = e + linear(W, "cond_embed", f64(cond))
    if cfg.cam_dim:
        e = e + linear(W, "cam_embed", f64(cam))
    return e


def patchify(z: np.ndarray, patch: Sequence[int]) -> np.ndarray:
    """[C,F,H,W] -> [N_v, C*pt*ph*pw]; token (f',h',w'), features ordered (c, a, i, j)."""
    c, f, h, w = z.shape
    pt, ph, pw = patch
    z7 = z.reshape(c, f // pt, pt, h // ph, ph, w // pw, pw)
    return z7.transpose(1, 3, 5, 0, 2, 4, 6).reshape((f // pt) * (h // ph) * (w // pw), c * pt * ph * pw)


def unpatchify(tok: np.ndarray, latent: Sequence[int], patch: Sequence[int]) -> np.ndarray:
    c, f, h, w = latent
    pt, ph, pw = patch
    t7 = tok.reshape(f // pt, h // ph, w // pw, c, pt, ph, pw)
    return t7.transpose(3, 0, 4, 1, 5, 2, 6).reshape(c, f, h, w)


def embed_tokens(W, cfg, z, text=None) -> np.ndarray:
    """Joint residual stream [N, D]: patch-embedded video rows, then projected text rows."""
    x = linear(W, "patch_embed", patchify(f64(z), cfg.patch))
    if cfg.text_tokens:
        x = np.concatenate([x, linear(W, "text_proj", f64(text))], axis=0)
    return x


def final_layer(W, cfg, x_video: np.ndarray, c_emb: np.ndarray) -> np.ndarray:
    mod = linear(W, "final.ada", silu(c_emb))
    shift, scale = np.split(mod, 2)
    out = linear(W, "final.lin", modulate(layer_norm(x_video), shift, scale))
    return unpatchify(out, cfg.latent, cfg.patch)


# ---------------------------------------------------------------------------
# blocks
# ---------------------------------------------------------------------------

def _select(rows, n):
    return np.arange(n) if rows is None else np.asarray(rows)


def seq_block(W, cfg, pre: str, x: np.ndarray, c_emb: np.ndarray, rows=None) -> np.ndarray:
    d = cfg.hidden
    sel = _select(rows, x.shape[0])
    sh1, sc1, g1, sh2, sc2, g2 = np.split(linear(W, pre + ".ada", silu(c_emb)), 6)
    h = modulate(layer_norm(x), sh1, sc1)
    ang = _angles(cfg)
    ridx = _rope_index(cfg, x.shape[0])
    k = _prep_qk(linear_rows(W, pre + ".qkv", h, d, 2 * d), cfg, ridx, ang)
    v = _heads(linear_rows(W, pre + ".qkv", h, 2 * d, 3 * d), cfg.heads)
    q = _prep_qk(linear_rows(W, pre + ".qkv", h[sel], 0, d), cfg, ridx[sel], ang)
    o = _merge(attention(q, k, v))
    xr = x[sel] + g1 * linear(W, pre + ".out", o)
    h2 = modulate(layer_norm(xr), sh2, sc2)
    return xr + g2 * linear(W, pre + ".fc2", gelu_tanh(linear(W, pre + ".fc1", h2)))


def dual_block(W, cfg, pre: str, x: np.ndarray, c_emb: np.ndarray, rows=None) -> np.ndarray:
    d, nv = cfg.hidden, cfg.n_video
    n = x.shape[0]
    sel = _select(rows, n)
    sc = silu(c_emb)
    mods = {s: np.split(linear(W, f"{pre}.{s}.ada", sc), 6) for s in ("vid", "txt")}
    spans = {"vid": (0, nv), "txt": (nv, n)}
    ang = _angles(cfg)
    ridx = _rope_index(cfg, n)
    ks, vs, hs = [], [], {}
    for s in ("vid", "txt"):
        a, b = spans[s]
        sh1, sc1 = mods[s][0], mods[s][1]
        hs[s] = modulate(layer_norm(x[a:b]), sh1, sc1)
        ks.append(linear_rows(W, f"{pre}.{s}.qkv", hs[s], d, 2 * d))
        vs.append(linear_rows(W, f"{pre}.{s}.qkv", hs[s], 2 * d, 3 * d))
    k = _prep_qk(np.concatenate(ks, 0), cfg, ridx, ang)
    v = _heads(np.concatenate(vs, 0), cfg.heads)
    out = np.empty((len(sel), d))
    for s in ("vid", "txt"):
        a, b = spans[s]
        m = (sel >= a) & (sel < b)
        if not m.any():
            continue
        rs = sel[m]
        q = _prep_qk(linear_rows(W, f"{pre}.{s}.qkv", hs[s][rs - a], 0, d), cfg, ridx[rs], ang)
        o = _merge(attention(q, k, v))
        sh1, sc1, g1, sh2, sc2, g2 = mods[s]
        xr = x[rs] + g1 * linear(W, f"{pre}.{s}.out", o)
        h2 = modulate(layer_norm(xr), sh2, sc2)
        out[m] = xr + g2 * linear(W, f"{pre}.{s}.fc2", gelu_tanh(linear(W, f"{pre}.{s}.fc1", h2)))
    return out


def single_block(W, cfg, pre: str, x: np.ndarray, c_emb: np.ndarray, rows=None) -> np.ndarray:
    d = cfg.hidden
    sel = _select(rows, x.shape[0])
    sh, scl, g = np.split(linear(W, pre + ".ada", silu(c_emb)), 3)
    h = modulate(layer_norm(x), sh, scl)
    ang = _angles(cfg)
    ridx = _rope_index(cfg, x.shape[0])
    k = _prep_qk(linear_rows(W, pre + ".lin1", h, d, 2 * d), cfg, ridx, ang)
    v = _heads(linear_rows(W, pre + ".lin1", h, 2 * d, 3 * d), cfg.heads)
    hr = h[sel]
    q = _prep_qk(linear_rows(W, pre + ".lin1", hr, 0, d), cfg, ridx[sel], ang)
    o = _merge(attention(q, k, v))
    mlp = gelu_tanh(linear_rows(W, pre + ".lin1", hr, 3 * d, W[pre + ".lin1.w"].shape[0]))
    return x[sel] + g * linear(W, pre + ".lin2", np.concatenate([o, mlp], axis=1))


def block_kind(cfg, block: int) -> str:
    if block < cfg.n_seq:
        return "seq"
    if block < cfg.n_seq + cfg.n_dual:
        return "dual"
    return "single"


def block_prefix(cfg, block: int) -> str:
    kind = block_kind(cfg, block)
    if kind == "seq":
        return f"seq.{block}"
    if kind == "dual":
        return f"dual.{block - cfg.n_seq}"
    return f"single.{block - cfg.n_seq - cfg.n_dual}"


def block_forward(W, cfg, block: int, x, c_emb, rows=None) -> np.ndarray:
    """One block of the global stack (sequential, then dual, then single)."""
    fn = {"seq": seq_block, "dual": dual_block, "single": single_block}[block_kind(cfg, block)]
    return fn(W, cfg, block_prefix(cfg, block), f64(x), f64(c_emb), rows)


def dit_forward(W, cfg, z, t: float, cond=None, text=None, cam=None) -> np.ndarray:
    """v = F_theta(z, t, c): [C,F,H,W] float64 velocity."""
    c_emb = cond_embedding(W, cfg, t, cond, cam)
    x = embed_tokens(W, cfg, z, text)
    for b in range(cfg.n_blocks):
        x = block_forward(W, cfg, b, x, c_emb)
    return final_layer(W, cfg, x[: cfg.n_video], c_emb)
