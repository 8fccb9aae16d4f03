"""ctypes binding of libwdc.so (include/wdc.h): argument marshalling only.

Every step of the rollout runs in the library's HIP kernels; PyTorch supplies
device memory (``torch.empty`` on the GPU) and the current stream. There is no
Python or CPU fallback: a missing library raises at load time.
"""
from __future__ import annotations

import ctypes as C
import math
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libwdc.so")

WDC_F32, WDC_BF16 = 0, 1
MODE_RISK, MODE_FORCED, MODE_ALL_EXACT, MODE_PERIODIC = 0, 1, 2, 3
SURROGATE_LIFTED, SURROGATE_SECANT = 0, 1
OBS_KERNEL, OBS_LINEAR = 0, 1
PRE_DECISION, POST_EXACT, POST_SURROGATE = 0, 1, 2
MAX_BANK = 8
# kernel timing classes, in the order of the WDC_T_* constants
TIMING_CLASSES = ("attention", "gemm", "stats", "observe", "exact_post", "psi", "norm")
STATUS = {0: "OK", 1: "E_ARG", 2: "E_SHAPE", 3: "E_DTYPE", 4: "E_ALIGN", 5: "E_WORKSPACE", 6: "E_STATE",
          7: "E_HIP", 8: "E_NONFINITE", 9: "E_UNSUPPORTED"}


class ModelDesc(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "dtype", "hidden", "heads", "head_dim", "mlp_ratio", "n_seq", "n_dual", "n_single", "cond_dim", "cam_dim",
        "text_tokens", "text_dim", "lat_c", "lat_f", "lat_h", "lat_w", "patch_t", "patch_h", "patch_w",
        "rope_t", "rope_h", "rope_w", "qk_norm", "max_batch")]


def desc_from_config(cfg, max_batch: int = 1) -> ModelDesc:
    """Model descriptor from any object with the workload fields (name, dtype, hidden, ...)."""
    d = ModelDesc()
    d.dtype = WDC_BF16 if cfg.dtype == "bf16" else WDC_F32
    d.hidden, d.heads, d.head_dim, d.mlp_ratio = cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp_ratio
    d.n_seq, d.n_dual, d.n_single = cfg.n_seq, cfg.n_dual, cfg.n_single
    d.cond_dim, d.cam_dim, d.text_tokens, d.text_dim = cfg.cond_dim, cfg.cam_dim, cfg.text_tokens, cfg.text_dim
    d.lat_c, d.lat_f, d.lat_h, d.lat_w = cfg.latent
    d.patch_t, d.patch_h, d.patch_w = cfg.patch
    d.rope_t, d.rope_h, d.rope_w = cfg.rope
    d.qk_norm = int(cfg.qk_norm)
    d.max_batch = max_batch
    return d


class Params(C.Structure):
    _fields_ = [("bank_capacity", C.c_int32), ("age_max", C.c_int32), ("n_min", C.c_int32), ("k_init", C.c_int32),
                ("k_ref", C.c_int32)] + [(n, C.c_double) for n in (
                    "theta_sim", "theta_q", "tau_in", "tau_obs", "gamma_q", "alpha_min", "alpha_max", "eps", "eps_nu",
                    "w_z", "w_age", "w_phase", "w_cam", "w_depth", "eta0", "beta_d", "eta_min", "eta_max",
                    "a_cam", "a_depth", "a_phase", "lam", "r0", "tau_risk")] + [(n, C.c_int32) for n in (
                    "period", "surrogate", "observation", "lift_condition", "impact_weight", "calibrate",
                    "support_constraint", "pad_")]


class StepLog(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("k", "exact", "bank", "support", "finite", "available", "slot", "pad_")] + [
        ("t", C.c_double), ("alpha", C.c_double), ("pi", C.c_double * MAX_BANK), ("kappa", C.c_double * MAX_BANK),
        ("sims_in", C.c_double * MAX_BANK)] + [(n, C.c_double) for n in (
            "d_z", "d_age", "d_phase", "p", "d_hat", "w", "r_cand", "margin", "sim_margin", "d_cf", "eta", "R")]

    def as_dict(self) -> dict:
        out = {}
        for name, _ in self._fields_:
            v = getattr(self, name)
            if name in ("pi", "kappa", "sims_in"):
                v = list(v)[: self.bank]
            out[name] = v
        return out


_lib = None


def load() -> C.CDLL:
    """Load libwdc.so (built in-tree by paper_2608_01845_amd.build); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_01845_amd.build`")
    lib = C.CDLL(LIB_PATH)
    vp, i32, i64, sz, dbl, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t, C.c_double, C.c_float
    sig = {
        "wdc_params_default": (None, [C.POINTER(Params)]),
        "wdc_create": (i32, [C.POINTER(ModelDesc), C.POINTER(Params), vp, C.POINTER(vp)]),
        "wdc_destroy": (i32, [vp]),
        "wdc_last_error": (C.c_char_p, [vp]),
        "wdc_weights_bytes": (sz, [vp]),
        "wdc_weight_count": (i32, [vp]),
        "wdc_weight_info": (i32, [vp, i32, C.POINTER(C.c_char_p), C.POINTER(i64), C.POINTER(i32), C.POINTER(sz)]),
        "wdc_bind_weights": (i32, [vp, vp, sz]),
        "wdc_init_weights_random": (i32, [vp, vp, sz, C.c_uint64, f32]),
        "wdc_workspace_bytes": (sz, [vp]),
        "wdc_bind_workspace": (i32, [vp, vp, sz]),
        "wdc_state_bytes": (sz, [vp]),
        "wdc_state_create": (i32, [vp, vp, sz, C.POINTER(vp)]),
        "wdc_state_reset": (i32, [vp, C.POINTER(f32)]),
        "wdc_state_destroy": (i32, [vp]),
        "wdc_state_bank_slot": (i32, [vp, i32, C.POINTER(vp), C.POINTER(i32)]),
        "wdc_cond_embed": (i32, [vp, dbl, vp, vp, vp]),
        "wdc_dit_block_forward": (i32, [vp, i32, vp, vp]),
        "wdc_dit_forward": (i32, [vp, vp, dbl, vp, vp, vp, vp]),
        "wdc_dit_forward_batch": (i32, [vp, i32, vp, dbl, vp, vp, vp, vp]),
        "wdc_scheduler_step": (i32, [vp, vp, vp, dbl, dbl, vp, i64]),
        "wdc_surrogate_step": (i32, [vp, vp, vp, i32, i32, vp, C.POINTER(StepLog)]),
        "wdc_surrogate_step_noalloc": (i32, [vp, vp, vp, i32, i32, vp, C.POINTER(StepLog)]),
        "wdc_risk_update": (i32, [vp, vp, i32, i32, i32, vp, vp, C.POINTER(StepLog)]),
        "wdc_rollout": (i32, [vp, vp, vp, i32, vp, vp, vp, i32, C.POINTER(C.c_uint8), vp, C.POINTER(C.c_uint8),
                              C.POINTER(StepLog)]),
        "wdc_rollout_batch": (i32, [vp, vp, i32, vp, i32, vp, vp, vp, i32, C.POINTER(C.c_uint8), vp,
                                    C.POINTER(C.c_uint8), C.POINTER(StepLog)]),
        "wdc_attn_pad": (i64, [i64]),
        "wdc_attention": (i32, [vp, vp, vp, vp, i64, vp, i64]),
        "wdc_attention_plan": (i32, [vp, i64, C.POINTER(i32), C.POINTER(i32)]),
        "wdc_linear": (i32, [vp, vp, i64, vp, vp, vp, i64, i64, i64, i64]),
        "wdc_set_timing": (i32, [vp, i32]),
        "wdc_timing": (i32, [vp, C.POINTER(dbl), C.POINTER(i64), C.POINTER(dbl)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def exported_symbols() -> List[str]:
    return [
        "wdc_params_default", "wdc_create", "wdc_destroy", "wdc_last_error", "wdc_weights_bytes", "wdc_weight_count",
        "wdc_weight_info", "wdc_bind_weights", "wdc_init_weights_random", "wdc_workspace_bytes", "wdc_bind_workspace",
        "wdc_state_bytes", "wdc_state_create", "wdc_state_reset", "wdc_state_destroy", "wdc_state_bank_slot",
        "wdc_cond_embed", "wdc_dit_block_forward", "wdc_dit_forward", "wdc_dit_forward_batch", "wdc_scheduler_step",
        "wdc_surrogate_step", "wdc_surrogate_step_noalloc", "wdc_risk_update", "wdc_rollout", "wdc_rollout_batch", "wdc_attn_pad", "wdc_attention", "wdc_attention_plan", "wdc_linear",
        "wdc_set_timing", "wdc_timing"]


class WdcError(RuntimeError):
    pass


def default_params(**overrides) -> Params:
    p = Params()
    load().wdc_params_default(C.byref(p))
    for k, v in overrides.items():
        setattr(p, k, v)
    return p


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _ptrs(ts):
    """Host array of device pointers of a list of tensors (None entries -> NULL), or None."""
    if ts is None:
        return None
    return (C.c_void_p * len(ts))(*[None if t is None else t.data_ptr() for t in ts])


def _torch():
    import torch
    return torch


class Context:
    """One model on one GPU stream. Device memory for weights, workspace and
    rollout state comes from torch allocations."""

    def __init__(self, cfg, params: Optional[Params] = None, device: str = "cuda:0", stream=None,
                 allocate_weights: bool = True, max_batch: int = 1):
        torch = _torch()
        self.lib = load()
        self.cfg = cfg
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.max_batch = max_batch
        self.desc = desc_from_config(cfg, max_batch)
        self.params = params if params is not None else default_params()
        h = C.c_void_p()
        self._check(self.lib.wdc_create(C.byref(self.desc), C.byref(self.params), C.c_void_p(self.stream.cuda_stream),
                                        C.byref(h)), None)
        self.h = h
        self.bf16 = cfg.dtype == "bf16"
        self.tdtype = torch.bfloat16 if self.bf16 else torch.float32
        ws = self.lib.wdc_workspace_bytes(h)
        self.workspace = torch.empty(max(ws, 256), dtype=torch.uint8, device=self.device)
        self._check(self.lib.wdc_bind_workspace(h, C.c_void_p(self.workspace.data_ptr()), self.workspace.numel()))
        self.weights = None
        nbytes = self.lib.wdc_weights_bytes(h)
        if allocate_weights and nbytes:
            self.weights = torch.zeros(nbytes, dtype=torch.uint8, device=self.device)
            self._check(self.lib.wdc_bind_weights(h, C.c_void_p(self.weights.data_ptr()), nbytes))

    # ---------------------------------------------------------------- plumbing
    def _check(self, status: int, h=-1):
        if status != 0:
            hh = self.h if h == -1 else h
            msg = self.lib.wdc_last_error(hh)
            raise WdcError(f"{STATUS.get(status, status)}: {msg.decode() if msg else ''}")

    def close(self):
        if getattr(self, "h", None):
            self.lib.wdc_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def n_tokens(self) -> int:
        c = self.cfg
        return c.n_video + c.text_tokens

    def weight_table(self) -> List[Tuple[str, Tuple[int, ...], int]]:
        out = []
        for i in range(self.lib.wdc_weight_count(self.h)):
            name = C.c_char_p()
            shape = (C.c_int64 * 2)()
            nd = C.c_int32()
            off = C.c_size_t()
            self._check(self.lib.wdc_weight_info(self.h, i, C.byref(name), shape, C.byref(nd), C.byref(off)))
            shp = (shape[0], shape[1]) if nd.value == 2 else (shape[0],)
            out.append((name.value.decode(), shp, off.value))
        return out

    def to_device(self, arr, dtype=None):
        """numpy -> device tensor in the model dtype (or ``dtype``); bf16 rounding is round-to-nearest-even."""
        torch = _torch()
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32))
        return t.to(self.device).to(dtype or self.tdtype).contiguous()

    def load_weights(self, named: Dict[str, np.ndarray], strict: bool = True):
        """Copy named tensors into the weight blob (name/shape from weight_table)."""
        torch = _torch()
        table = self.weight_table()
        seen = 0
        esz = 2 if self.bf16 else 4
        for name, shape, off in table:
            if name not in named:
                if strict:
                    raise KeyError(f"missing weight {name}")
                continue
            a = np.asarray(named[name], dtype=np.float32)
            if tuple(a.shape) != tuple(shape):
                raise ValueError(f"{name}: shape {a.shape} != {shape}")
            dev = self.to_device(a).reshape(-1).view(torch.uint8)
            self.weights[off: off + a.size * esz].copy_(dev)
            seen += 1
        return seen

    def bind_weights(self, blob):
        """Bind an existing weight blob (a uint8 device tensor, e.g. another context's
        ``weights`` for the same model) instead of this context's own."""
        self._check(self.lib.wdc_bind_weights(self.h, C.c_void_p(blob.data_ptr()), blob.numel()))
        self.weights = blob

    def init_random_weights(self, seed: int = 0, std: float = 0.02):
        self._check(self.lib.wdc_init_weights_random(self.h, C.c_void_p(self.weights.data_ptr()),
                                                     self.weights.numel(), seed, std))

    # ---------------------------------------------------------------- denoiser
    def cond_embed(self, t: float, cond=None, cam=None, out=None):
        torch = _torch()
        out = out if out is not None else torch.empty(self.cfg.hidden, dtype=torch.float32, device=self.device)
        self._check(self.lib.wdc_cond_embed(self.h, t, _ptr(cond), _ptr(cam), _ptr(out)))
        return out

    def block_forward(self, block: int, x, cemb):
        """In place on x [N, D] float32."""
        self._check(self.lib.wdc_dit_block_forward(self.h, block, _ptr(x), _ptr(cemb)))
        return x

    def forward(self, z, t: float, cond=None, text=None, cam=None, out=None):
        torch = _torch()
        out = out if out is not None else torch.empty_like(z)
        self._check(self.lib.wdc_dit_forward(self.h, _ptr(z), t, _ptr(cond), _ptr(text), _ptr(cam), _ptr(out)))
        return out

    def forward_batch(self, zs, t: float, conds=None, texts=None, cams=None, outs=None):
        """F_theta of len(zs) samples at one t in one batched pass; lists of tensors."""
        torch = _torch()
        b = len(zs)
        outs = outs if outs is not None else [torch.empty_like(z) for z in zs]
        self._check(self.lib.wdc_dit_forward_batch(self.h, b, _ptrs(zs), t, _ptrs(conds), _ptrs(texts), _ptrs(cams),
                                                   _ptrs(outs)))
        return outs

    def scheduler_step(self, z, v, t_cur: float, t_next: float, out=None):
        torch = _torch()
        out = out if out is not None else torch.empty_like(z)
        self._check(self.lib.wdc_scheduler_step(self.h, _ptr(z), _ptr(v), t_cur, t_next, _ptr(out), z.numel()))
        return out

    def attention(self, q, k, vt, n: int, out, ldo: int):
        self._check(self.lib.wdc_attention(self.h, _ptr(q), _ptr(k), _ptr(vt), n, _ptr(out), ldo))
        return out

    def attn_pad(self, n: int) -> int:
        return self.lib.wdc_attn_pad(n)

    def attention_plan(self, n: int):
        """(query blocks per head over all keys, key ranges of each remaining block)."""
        qb, ks = C.c_int32(), C.c_int32()
        self._check(self.lib.wdc_attention_plan(self.h, n, C.byref(qb), C.byref(ks)))
        return qb.value, ks.value

    def linear(self, a, w, bias, out, m: int, n: int, k: int, lda: int = None, ldc: int = None):
        self._check(self.lib.wdc_linear(self.h, _ptr(a), lda or k, _ptr(w), _ptr(bias), _ptr(out), ldc or n, m, n, k))
        return out

    def set_timing(self, on: bool):
        self._check(self.lib.wdc_set_timing(self.h, int(on)))

    def timing(self):
        n = len(TIMING_CLASSES)
        ms, cnt, work = (C.c_double * n)(), (C.c_int64 * n)(), (C.c_double * n)()
        self._check(self.lib.wdc_timing(self.h, ms, cnt, work))
        return {name: (ms[i], cnt[i], work[i]) for i, name in enumerate(TIMING_CLASSES)}

    # ---------------------------------------------------------------- surrogate, risk, rollout
    def new_state(self) -> "State":
        return State(self)

    def rollout(self, state: "State", z, steps: int, cond=None, text=None, cam=None, mode: int = MODE_RISK,
                forced: Optional[Sequence[int]] = None, replay_v=None):
        sched = (C.c_uint8 * steps)()
        logs = (StepLog * steps)()
        fz = None
        if forced is not None:
            fz = (C.c_uint8 * steps)(*[int(x) for x in forced])
        self._check(self.lib.wdc_rollout(self.h, state.h, _ptr(z), steps, _ptr(cond), _ptr(text), _ptr(cam), mode,
                                         fz, _ptr(replay_v), sched, logs))
        return list(sched), [l.as_dict() for l in logs]

    def rollout_batch(self, states: Sequence["State"], zs, steps: int, conds=None, texts=None, cams=None,
                      mode: int = MODE_RISK, forced: Optional[Sequence[Sequence[int]]] = None, replay_vs=None):
        """len(zs) rollouts at once (each latent updated in place); per-sample
        schedules [B][S] and logs [B][S]."""
        b = len(zs)
        sched = (C.c_uint8 * (b * steps))()
        logs = (StepLog * (b * steps))()
        fz = None
        if forced is not None:
            fz = (C.c_uint8 * (b * steps))(*[int(x) for row in forced for x in row])
        st = (C.c_void_p * b)(*[s.h.value for s in states])
        self._check(self.lib.wdc_rollout_batch(self.h, st, b, _ptrs(zs), steps, _ptrs(conds), _ptrs(texts),
                                               _ptrs(cams), mode, fz, _ptrs(replay_vs), sched, logs))
        return ([list(sched[i * steps:(i + 1) * steps]) for i in range(b)],
                [[logs[i * steps + k].as_dict() for k in range(steps)] for i in range(b)])

    def surrogate_step(self, state: "State", z, k: int, steps: int, zhat) -> dict:
        log = StepLog()
        self._check(self.lib.wdc_surrogate_step(self.h, state.h, _ptr(z), k, steps, _ptr(zhat), C.byref(log)))
        return log.as_dict()

    def surrogate_step_noalloc(self, state: "State", z, k: int, steps: int, zhat) -> dict:
        """surrogate_step with the statistics scratch in the library's fixed device array."""
        log = StepLog()
        self._check(self.lib.wdc_surrogate_step_noalloc(self.h, state.h, _ptr(z), k, steps, _ptr(zhat),
                                                        C.byref(log)))
        return log.as_dict()

    def risk_update(self, state: "State", phase: int, k: int, steps: int, z_cur=None, z_next=None) -> dict:
        log = StepLog()
        self._check(self.lib.wdc_risk_update(self.h, state.h, phase, k, steps, _ptr(z_cur), _ptr(z_next),
                                             C.byref(log)))
        return log.as_dict()


class State:
    """Rollout state (bank, anchor, history, risk); device memory from torch."""

    def __init__(self, ctx: Context):
        torch = _torch()
        self.ctx = ctx
        n = ctx.lib.wdc_state_bytes(ctx.h)
        self.mem = torch.empty(n, dtype=torch.uint8, device=ctx.device)
        h = C.c_void_p()
        ctx._check(ctx.lib.wdc_state_create(ctx.h, C.c_void_p(self.mem.data_ptr()), n, C.byref(h)))
        self.h = h

    def reset(self, cam: Optional[np.ndarray] = None):
        arr = None
        if cam is not None:
            c = np.ascontiguousarray(cam, dtype=np.float32)
            arr = c.ctypes.data_as(C.POINTER(C.c_float))
        self.ctx._check(self.ctx.lib.wdc_state_reset(self.h, arr))

    def bank_slot(self, i: int):
        p = C.c_void_p()
        ins = C.c_int32()
        self.ctx._check(self.ctx.lib.wdc_state_bank_slot(self.h, i, C.byref(p), C.byref(ins)))
        return p.value, ins.value

    def close(self):
        if getattr(self, "h", None):
            self.ctx.lib.wdc_state_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
