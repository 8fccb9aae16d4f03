"""Parity check run in a child process with one comparison switch set.

The library reads its comparison switches (WDC_GEMM_VARIANT, WDC_ATTN_VARIANT,
...) once per process, so tests/test_gpu_switches.py starts this script with
the switch in its environment. It checks the bf16 GEMM on products that take
the 256 x 256 block tiles, or the bf16 attention at hd 64 and 128, against the oracle
and exits non-zero on a mismatch.
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import dit  # noqa: E402
from tests.gpu_util import context, rel_l2, small_cfg, torch_cuda  # noqa: E402


def check_gemm() -> float:
    torch = torch_cuda()
    cfg = synth.get_config("mid")
    ctx = context(cfg, weights=False)
    worst = 0.0
    for m, n, k in ((1000, 512, 3072), (700, 2048, 256), (2100, 4096, 128), (513, 768, 1024)):
        rng = np.random.default_rng(m * 7 + n)
        a = synth.stored(rng.standard_normal((m, k)), cfg.dtype)
        w = synth.stored(rng.standard_normal((n, k)) * 0.05, cfg.dtype)
        b = synth.stored(rng.standard_normal(n) * 0.1, cfg.dtype)
        out = torch.empty((m, n), dtype=ctx.tdtype, device="cuda")
        ctx.linear(ctx.to_device(a), ctx.to_device(w), ctx.to_device(b), out, m, n, k)
        err = rel_l2(out.float().cpu().numpy(), dit.linear({"l.w": w, "l.b": b}, "l", a.astype(np.float64)))
        print(f"gemm m {m} n {n} k {k}: rel_l2 {err:.2e}", flush=True)
        worst = max(worst, err)
    return worst


def check_attention() -> float:
    from tests.test_gpu_kernels import _attn_inputs
    torch = torch_cuda()
    worst = 0.0
    for hd in (64, 128):
        cfg = small_cfg("bf16", head_dim=hd)
        ctx = context(cfg, weights=False)
        heads = cfg.heads
        # 1, 2, 7, 8, 11 and 18 key tiles (the hd 64 two-phase form loads six ahead over eight slots)
        for n in ((61, 100, 385, 449, 700, 1111) if hd == 64 else (61, 100, 700, 1111)):
            (q, k, v), (qd, kd, vd) = _attn_inputs(ctx, heads, hd, n, seed=n, bf16=True)
            out = torch.zeros((n, heads * hd), dtype=torch.bfloat16, device="cuda")
            ctx.attention(qd, kd, vd, n, out, heads * hd)
            ref = dit.attention(q, k, v).transpose(1, 0, 2).reshape(n, heads * hd)
            err = rel_l2(out.float().cpu().numpy(), ref)
            print(f"attention hd {hd} n {n}: rel_l2 {err:.2e}", flush=True)
            worst = max(worst, err)
    return worst


if __name__ == "__main__":
    kind = sys.argv[1]
    # bf16 output rounding dominates both (the same bounds as the default-path tests)
    worst, tol = (check_gemm(), 4e-3) if kind == "gemm" else (check_attention(), 1e-2)
    print(f"worst {worst:.2e} (tolerance {tol:.0e})", flush=True)
    sys.exit(0 if worst <= tol else 1)
