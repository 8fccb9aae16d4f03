"""The q/k/v projection with per-head RMSNorm, RoPE and the attention layouts
fused into the GEMM epilogue, against the plain GEMM followed by the separate
preparation kernels (GPU). Both round the projection to bf16 once and then
apply the same float32 arithmetic, so the blocks must agree bit for bit; the
oracle comparison of the fused path is in the block, forward and full-size
tests."""
import os

import numpy as np
import pytest

import synth
from oracle import dit
from tests.gpu_util import TOL_BF16_BLOCK, rel_l2, small_cfg, torch_cuda

pytestmark = pytest.mark.gpu


def _pair(cfg, max_batch=1):
    """(fused, separate) contexts sharing one weight blob. These products are
    too small to fill a dispatch round of 256 x 256 tiles, which would send
    them to the 128 x 128 tiles and the separate kernels: the fused context
    keeps the tile size the shape selects (WDC_FILL_TILES=0)."""
    import paper_2608_01845_amd as wdc
    os.environ["WDC_FILL_TILES"] = "0"
    try:
        fused = wdc.Context(cfg, max_batch=max_batch)
    finally:
        del os.environ["WDC_FILL_TILES"]
    fused.load_weights(synth.gen_weights(cfg))
    os.environ["WDC_FUSE_QKV"] = "0"
    try:
        sep = wdc.Context(cfg, max_batch=max_batch, allocate_weights=False)
    finally:
        del os.environ["WDC_FUSE_QKV"]
    sep.bind_weights(fused.weights)
    return fused, sep


@pytest.mark.parametrize("head_dim,rope", [(64, True), (128, True), (64, False), (128, False)])
def test_fused_qkv_blocks_equal_separate_preparation(head_dim, rope):
    """560 video + 21 text tokens: the sequential and single blocks and the
    dual block's video stream take the fused epilogue (the 21 text rows of the
    dual block stay on the separate kernels); the last 256-row tile is partial
    and its last group of 16 tokens incomplete. Without rotary dimensions the
    epilogue takes its form without rotation-table reads."""
    torch = torch_cuda()
    cfg = small_cfg("bf16", head_dim=head_dim, latent=(16, 4, 20, 28), **({} if rope else {"rope": (0, 0, 0)}))
    fused, sep = _pair(cfg)
    x = synth.gen_block_input(cfg)
    c = torch.from_numpy(synth.gen_cemb(cfg)).cuda()
    W = synth.gen_weights(cfg)
    for b in range(cfg.n_blocks):
        xf = torch.from_numpy(x).cuda()
        xs = xf.clone()
        fused.block_forward(b, xf, c)
        sep.block_forward(b, xs, c)
        diff = float((xf - xs).abs().max())
        print(f"hd {head_dim} block {b}: fused vs separate max |diff| {diff:.3e}")
        assert torch.equal(xf, xs), (b, diff)
        err = rel_l2(xf.cpu().numpy(), dit.block_forward(W, cfg, b, x, synth.gen_cemb(cfg)))
        print(f"hd {head_dim} block {b} ({dit.block_kind(cfg, b)}): fused == separate, oracle rel_l2 {err:.2e}")
        assert err <= TOL_BF16_BLOCK


def test_fused_qkv_batched_forward_equals_separate_preparation():
    """Two samples in one product: 581-token samples, so a 256-row tile holds
    rows of both samples and the first token of most tiles is not 16-aligned
    (the element-wise V^T path)."""
    torch = torch_cuda()
    cfg = small_cfg("bf16", head_dim=64, latent=(16, 4, 20, 28))
    fused, sep = _pair(cfg, max_batch=2)
    zs = [torch.from_numpy(synth.gen_tensor(s, "z", cfg.latent)).cuda() for s in (1, 2)]
    inp = synth.gen_inputs(cfg)
    conds = [fused.to_device(inp["cond"])] * 2
    texts = [fused.to_device(inp["text"])] * 2
    cams = [fused.to_device(inp["cam"])] * 2
    vf = fused.forward_batch(zs, 0.4, conds, texts, cams)
    vs = sep.forward_batch(zs, 0.4, conds, texts, cams)
    for a, b in zip(vf, vs):
        print("batched forward: fused vs separate max |diff|", float((a - b).abs().max()))
        assert torch.isfinite(a).all() and torch.equal(a, b)


def test_fill_tiles_mid_forward_bitwise_equal():
    """The mid-size forward (2,688 tokens, D = 1,024) with its products on 128 x
    128 tiles and the separate q/k/v preparation (the default: no product fills
    a dispatch round of 256 x 256 tiles) against the 256 x 256 tiles and the
    fused epilogue: both sum every output over K in the same order and apply
    the same float32 arithmetic afterwards, so the velocities agree bit for bit."""
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    cfg = synth.get_config("mid")
    fill = wdc.Context(cfg)
    fill.init_random_weights(seed=5, std=0.02)
    os.environ["WDC_FILL_TILES"] = "0"
    try:
        shape = wdc.Context(cfg, allocate_weights=False)
    finally:
        del os.environ["WDC_FILL_TILES"]
    shape.bind_weights(fill.weights)
    inp = synth.gen_inputs(cfg)
    z = torch.from_numpy(inp["z_T"]).cuda()
    cond = fill.to_device(inp["cond"])
    a = fill.forward(z, 0.7, cond)
    b = shape.forward(z, 0.7, cond)
    print("mid forward: 128 x 128 + separate vs 256 x 256 + fused max |diff|", float((a - b).abs().max()))
    assert torch.isfinite(a).all() and torch.equal(a, b)
