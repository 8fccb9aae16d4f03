"""Seeded synthetic inputs for the WorldDynCache denoising rollout.

This module is the only code shared by the CPU oracle and the GPU path. It
holds workload shapes and random-number generation, and none of the method's
arithmetic: no transformer, no scheduler, no surrogate, no risk estimator.

Every tensor is drawn from its own stream. The stream of tensor ``name`` in a
workload with seed ``s`` is ``numpy.random.PCG64(SeedSequence([s, crc32(name)]))``
and values are ``std * standard_normal`` in float64, then rounded once to the
workload's storage type (float32, or bfloat16 with round-to-nearest-even).

Workloads (the paper's denoisers are not public, so these are random-init
stand-ins shaped like its 5B- and 13B-class video world models):

* ``tiny``   2 sequential blocks, D=256, 4x64 heads, fp32, 16x4x16x16 latent.
* ``mid``    8 sequential blocks, D=1024, 16x64 heads, bf16, 16x7x32x48 latent.
* ``5b``     30 sequential blocks over a joint [video; 226 text] sequence,
             D=3072, 48x64 heads, camera vector, bf16, 16x13x60x90 latent.
* ``13b``    20 dual-stream + 40 single-stream blocks, D=3072, 24x128 heads,
             256 text tokens, bf16, 16x33x68x120 latent.
* ``stress`` one single-stream block at 16x33x90x160 (118800 tokens), and
             the surrogate/risk kernels standalone on that latent.
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field, replace
from typing import Dict, Iterable, List, Optional, Tuple

import numpy as np

__all__ = [
    "ModelConfig", "CONFIGS", "get_config", "weight_specs", "gen_tensor",
    "gen_weights", "gen_inputs", "round_bf16", "to_bf16_bits", "from_bf16_bits",
    "stream", "bank_inputs", "stored",
]


@dataclass(frozen=True)
class ModelConfig:
    name: str
    dtype: str                      # "f32" or "bf16": storage/compute type of weights and activations
    hidden: int                     # D
    heads: int
    head_dim: int
    mlp_ratio: int = 4
    n_seq: int = 0                  # sequential blocks (shared weights over the joint sequence)
    n_dual: int = 0                 # dual-stream blocks (per-stream weights, joint attention)
    n_single: int = 0               # single-stream blocks (fused linear1/linear2)
    cond_dim: int = 0               # pooled condition vector length
    cam_dim: int = 0                # camera/geometry vector length (0: none)
    text_tokens: int = 0
    text_dim: int = 0
    latent: Tuple[int, int, int, int] = (16, 4, 16, 16)   # C, F, H, W
    patch: Tuple[int, int, int] = (1, 2, 2)                # pt, ph, pw
    rope: Tuple[int, int, int] = (16, 24, 24)              # rotary dims for (t, h, w); sum = head_dim
    qk_norm: bool = True
    steps: int = 8
    seed: int = 0

    # derived shapes ---------------------------------------------------------
    @property
    def grid(self) -> Tuple[int, int, int]:
        c, f, h, w = self.latent
        pt, ph, pw = self.patch
        return (f // pt, h // ph, w // pw)

    @property
    def n_video(self) -> int:
        g = self.grid
        return g[0] * g[1] * g[2]

    @property
    def n_tokens(self) -> int:
        return self.n_video + self.text_tokens

    @property
    def patch_dim(self) -> int:
        c = self.latent[0]
        pt, ph, pw = self.patch
        return c * pt * ph * pw

    @property
    def numel(self) -> int:
        c, f, h, w = self.latent
        return c * f * h * w

    @property
    def n_blocks(self) -> int:
        return self.n_seq + self.n_dual + self.n_single

    def flops_per_forward(self) -> float:
        """Dense matrix-core work of one forward: 24*N*D^2 + 4*N^2*D per block,
        with N the joint sequence length and single blocks counted at 7D/5D widths."""
        n, d = self.n_tokens, self.hidden
        per_seq = 24.0 * n * d * d + 4.0 * n * n * d
        # single block: linear1 (D -> 7D) + linear2 (5D -> D) = 24 N D^2 as well
        return (self.n_seq + self.n_dual + self.n_single) * per_seq


_BASE = dict(mlp_ratio=4, patch=(1, 2, 2), qk_norm=True)

CONFIGS: Dict[str, ModelConfig] = {
    "tiny": ModelConfig(name="tiny", dtype="f32", hidden=256, heads=4, head_dim=64,
                        n_seq=2, cond_dim=256, latent=(16, 4, 16, 16),
                        rope=(16, 24, 24), steps=8, seed=0, **_BASE),
    "mid": ModelConfig(name="mid", dtype="bf16", hidden=1024, heads=16, head_dim=64,
                       n_seq=8, cond_dim=1024, latent=(16, 7, 32, 48),
                       rope=(16, 24, 24), steps=20, seed=1, **_BASE),
    "5b": ModelConfig(name="5b", dtype="bf16", hidden=3072, heads=48, head_dim=64,
                      n_seq=30, cond_dim=4096, cam_dim=3072, text_tokens=226, text_dim=4096,
                      latent=(16, 13, 60, 90), rope=(16, 24, 24), steps=50, seed=2, **_BASE),
    "13b": ModelConfig(name="13b", dtype="bf16", hidden=3072, heads=24, head_dim=128,
                       n_dual=20, n_single=40, cond_dim=4096, text_tokens=256, text_dim=4096,
                       latent=(16, 33, 68, 120), rope=(16, 56, 56), steps=50, seed=3, **_BASE),
    "stress": ModelConfig(name="stress", dtype="bf16", hidden=3072, heads=24, head_dim=128,
                          n_single=1, cond_dim=4096, latent=(16, 33, 90, 160),
                          rope=(16, 56, 56), steps=50, seed=4, **_BASE),
}


def get_config(name: str, **overrides) -> ModelConfig:
    cfg = CONFIGS[name]
    return replace(cfg, **overrides) if overrides else cfg


# ---------------------------------------------------------------------------
# parameter inventory (names and shapes only)
# ---------------------------------------------------------------------------

def weight_specs(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    """Every parameter tensor of the synthetic DiT, in storage order.
    Linear weights are [out, in] (input features contiguous), biases [out]."""
    d, p = cfg.hidden, cfg.patch_dim
    f = cfg.mlp_ratio * d
    specs: List[Tuple[str, Tuple[int, ...]]] = []

    def lin(name, out, inp):
        specs.append((name + ".w", (out, inp)))
        specs.append((name + ".b", (out,)))

    lin("t_embed.fc1", d, 256)
    lin("t_embed.fc2", d, d)
    if cfg.cond_dim:
        lin("cond_embed", d, cfg.cond_dim)
    if cfg.cam_dim:
        lin("cam_embed", d, cfg.cam_dim)
    if cfg.text_tokens:
        lin("text_proj", d, cfg.text_dim)
    lin("patch_embed", d, p)
    for i in range(cfg.n_seq):
        pre = f"seq.{i}"
        lin(pre + ".ada", 6 * d, d)
        lin(pre + ".qkv", 3 * d, d)
        lin(pre + ".out", d, d)
        lin(pre + ".fc1", f, d)
        lin(pre + ".fc2", d, f)
    for i in range(cfg.n_dual):
        for s in ("vid", "txt"):
            pre = f"dual.{i}.{s}"
            lin(pre + ".ada", 6 * d, d)
            lin(pre + ".qkv", 3 * d, d)
            lin(pre + ".out", d, d)
            lin(pre + ".fc1", f, d)
            lin(pre + ".fc2", d, f)
    for i in range(cfg.n_single):
        pre = f"single.{i}"
        lin(pre + ".ada", 3 * d, d)
        lin(pre + ".lin1", 3 * d + f, d)
        lin(pre + ".lin2", d, d + f)
    lin("final.ada", 2 * d, d)
    lin("final.lin", p, d)
    return specs


def block_prefix(cfg: ModelConfig, block: int) -> str:
    """Global block index -> parameter prefix: sequential, then dual, then single."""
    if block < cfg.n_seq:
        return f"seq.{block}"
    block -= cfg.n_seq
    if block < cfg.n_dual:
        return f"dual.{block}"
    block -= cfg.n_dual
    if block < cfg.n_single:
        return f"single.{block}"
    raise IndexError("block index out of range")


# ---------------------------------------------------------------------------
# rounding helpers (storage types of the inputs)
# ---------------------------------------------------------------------------

def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float -> bfloat16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Values of ``x`` rounded to bfloat16, returned as float32."""
    return from_bf16_bits(to_bf16_bits(x))


def stored(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round to the storage type; float32 array either way."""
    x = np.asarray(x, dtype=np.float32)
    return round_bf16(x) if dtype == "bf16" else x


# ---------------------------------------------------------------------------
# streams
# ---------------------------------------------------------------------------

def stream(seed: int, name: str) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), zlib.crc32(name.encode())])))


def gen_tensor(seed: int, name: str, shape: Iterable[int], std: float = 1.0,
               dtype: str = "f32", mean: float = 0.0) -> np.ndarray:
    g = stream(seed, name)
    x = g.standard_normal(tuple(shape), dtype=np.float64) * std + mean
    return stored(x, dtype)


WEIGHT_STD = 0.02


def gen_weights(cfg: ModelConfig, names: Optional[Iterable[str]] = None,
                std: float = WEIGHT_STD) -> Dict[str, np.ndarray]:
    """Seeded parameters (weights and biases ~ N(0, std)), float32 arrays holding
    values of the workload's storage type. ``names``: subset (prefix match)."""
    specs = weight_specs(cfg)
    want = None if names is None else tuple(names)
    out = {}
    for n, shp in specs:
        if want is not None and not any(n == w or n.startswith(w + ".") for w in want):
            continue
        out[n] = gen_tensor(cfg.seed, n, shp, std=std, dtype=cfg.dtype)
    return out


def gen_inputs(cfg: ModelConfig) -> Dict[str, np.ndarray]:
    """z_T (fp32 state), pooled condition, text features and camera vector."""
    d = {}
    d["z_T"] = gen_tensor(cfg.seed, "z_T", cfg.latent, dtype="f32")
    if cfg.cond_dim:
        d["cond"] = gen_tensor(cfg.seed, "cond", (cfg.cond_dim,), dtype=cfg.dtype)
    if cfg.cam_dim:
        d["cam"] = gen_tensor(cfg.seed, "cam", (cfg.cam_dim,), dtype=cfg.dtype)
    if cfg.text_tokens:
        d["text"] = gen_tensor(cfg.seed, "text", (cfg.text_tokens, cfg.text_dim), dtype=cfg.dtype)
    return d


def gen_cemb(cfg: ModelConfig, name: str = "c_emb") -> np.ndarray:
    """A conditioning vector for standalone block tests, ~N(0,1), fp32."""
    return gen_tensor(cfg.seed, name, (cfg.hidden,), dtype="f32")


def gen_block_input(cfg: ModelConfig, name: str = "x_block") -> np.ndarray:
    """Residual-stream input [N, D] for standalone block tests, ~N(0,1), fp32."""
    return gen_tensor(cfg.seed, name, (cfg.n_tokens, cfg.hidden), dtype="f32")


def gen_replay_velocities(cfg: ModelConfig, steps: Optional[int] = None) -> np.ndarray:
    """Velocities [S, C, F, H, W] standing in for F_theta at every step (replay mode).
    A smooth shared direction plus per-step noise, so consecutive exact increments
    are correlated the way a denoising trajectory's are."""
    s = cfg.steps if steps is None else steps
    base = gen_tensor(cfg.seed, "replay_base", cfg.latent, dtype="f32").astype(np.float64)
    out = np.empty((s,) + tuple(cfg.latent), dtype=np.float32)
    for k in range(s):
        noise = stream(cfg.seed, f"replay_noise.{k}").standard_normal(cfg.latent)
        out[k] = (base + 0.3 * noise).astype(np.float32)
    return out


def bank_inputs(cfg: ModelConfig, m: int = 4) -> Dict[str, np.ndarray]:
    """Standalone surrogate/risk workload: a latent, ``m`` stored exact outputs
    that are small perturbations of it (a trajectory-like bank), ``m`` velocities."""
    z = gen_tensor(cfg.seed, "bank_z", cfg.latent, dtype="f32").astype(np.float64)
    outs = np.stack([(z + 0.1 * stream(cfg.seed, f"bank_out.{i}").standard_normal(cfg.latent)).astype(np.float32)
                     for i in range(m)])
    vel = np.stack([gen_tensor(cfg.seed, f"bank_v.{i}", cfg.latent, dtype="f32") for i in range(m)])
    anchor = (z + 0.05 * stream(cfg.seed, "bank_anchor").standard_normal(cfg.latent)).astype(np.float32)
    return {"z": z.astype(np.float32), "z_out": outs, "v": vel, "z_a": anchor}
