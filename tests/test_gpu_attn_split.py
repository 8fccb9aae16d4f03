"""The attention's key-range split of the last, partly filled dispatch round
(GPU): query blocks of that round run as several blocks over disjoint key
ranges, each leaving its unnormalised rows, reference maxima and row sums in
scratch, and a second launch combines them. Checked against the oracle at the
attention tolerances of test_gpu_kernels.py (1e-2 relative L2, 3e-2 per row
and head), with the split forced (WDC_ATTN_SPLITS) at sizes the oracle
finishes in seconds, and against the unsplit kernel on the same inputs."""
import os

import numpy as np
import pytest

from oracle import dit
from tests.gpu_util import context, rel_l2, row_rel_l2, small_cfg, torch_cuda
from tests.test_gpu_kernels import ROW_TOL_ATTN_BF16, _attn_inputs

pytestmark = pytest.mark.gpu

# a latent large enough that the projection area of the workspace (the
# split's scratch) holds every split below
LATENT = (16, 8, 64, 64)


def _ctx(head_dim, splits, **kw):
    os.environ["WDC_ATTN_SPLITS"] = str(splits)
    try:
        return context(small_cfg("bf16", head_dim=head_dim, latent=LATENT, **kw), weights=False)
    finally:
        del os.environ["WDC_ATTN_SPLITS"]


def _run(ctx, inputs, n, heads, hd):
    torch = torch_cuda()
    qd, kd, vd = inputs
    out = torch.zeros((n, heads * hd), dtype=torch.bfloat16, device="cuda")
    ctx.attention(qd, kd, vd, n, out, heads * hd)
    return out


@pytest.mark.parametrize("head_dim,n,splits", [
    (64, 65, 2), (64, 300, 3), (64, 1400, 4), (64, 900, 8), (128, 130, 2), (128, 777, 3), (128, 1400, 5)])
def test_split_round_matches_oracle(head_dim, n, splits):
    """Few heads and short sequences: every query block is in the partial
    round, so all of them run split (ranges of 1-4 key tiles at the short
    lengths, the last one partial), and match the oracle."""
    ctx = _ctx(head_dim, splits)
    heads = 256 // head_dim
    qb_main, ks = ctx.attention_plan(n)
    tiles = (n + 63) // 64
    assert qb_main == 0 and ks == min(splits, tiles), (qb_main, ks)
    (q, k, v), dev = _attn_inputs(ctx, heads, head_dim, n, seed=n + splits, bf16=True)
    got = _run(ctx, dev, n, heads, head_dim).float().cpu().numpy()
    ref = dit.attention(q, k, v).transpose(1, 0, 2).reshape(n, heads * head_dim)
    err = rel_l2(got, ref)
    rerr = row_rel_l2(got.reshape(n, heads, head_dim), ref.reshape(n, heads, head_dim))
    print(f"hd {head_dim} n {n} ranges {ks}: rel_l2 {err:.2e}, worst row {rerr:.2e}")
    assert err <= 1e-2 and rerr <= ROW_TOL_ATTN_BF16


@pytest.mark.parametrize("head_dim", [64, 128])
def test_whole_rounds_and_split_round_in_one_launch(head_dim):
    """8 heads (blocks of one head on one XCD) and 8,492 tokens: 34 query
    blocks per head, of which 32 x 8 = 256 fill one whole round over all keys
    and the other 2 x 8 run as 4 key ranges each. Sampled query rows of both
    parts against the oracle; the whole output against the unsplit kernel;
    two calls in a row give the same bits."""
    torch = torch_cuda()
    heads, n = 8, 8492
    kw = dict(heads=heads, hidden=heads * head_dim)
    split, whole = _ctx(head_dim, 4, **kw), _ctx(head_dim, 1, **kw)
    assert split.attention_plan(n) == (32, 4) and whole.attention_plan(n) == (34, 1)
    (q, k, v), dev = _attn_inputs(split, heads, head_dim, n, seed=7, bf16=True)
    a = _run(split, dev, n, heads, head_dim)
    b = _run(split, dev, n, heads, head_dim)
    c = _run(whole, dev, n, heads, head_dim)
    assert torch.equal(a, b)
    got, unsplit = a.float().cpu().numpy(), c.float().cpu().numpy()
    rows = np.r_[0:3, 4000:4003, 32 * 256 - 2:32 * 256 + 2, n - 3:n]
    ref = dit.attention(q[:, rows], k, v).transpose(1, 0, 2).reshape(len(rows), heads * head_dim)
    err = rel_l2(got[rows], ref)
    rerr = row_rel_l2(got[rows].reshape(-1, heads, head_dim), ref.reshape(-1, heads, head_dim))
    tail = slice(32 * 256, n)
    diff = rel_l2(got[tail], unsplit[tail])
    print(f"hd {head_dim}: sampled rows rel_l2 {err:.2e}, worst row {rerr:.2e}; split round vs unsplit {diff:.2e}")
    assert err <= 1e-2 and rerr <= ROW_TOL_ATTN_BF16
    # the rows over all keys are the same kernel and the same arithmetic
    assert np.array_equal(got[:32 * 256], unsplit[:32 * 256])
    # the split rows differ from the unsplit ones by the bf16 roundings only
    assert diff <= 5e-3


def test_batched_forward_with_split_round():
    """A two-sample batched forward of the mid-size model (2 x 16 heads of 11
    query blocks: 8 per head fill whole rounds, the other 3 x 32 run as 3 key
    ranges, forced) against the same forward with the split switched off, and
    one sample against the oracle."""
    torch = torch_cuda()
    import paper_2608_01845_amd as wdc
    import synth
    from tests.gpu_util import TOL_BF16_FINAL
    from tests.test_gpu_batch import inputs
    cfg = synth.get_config("mid")
    ctxs = []
    for splits in (3, 1):
        os.environ["WDC_ATTN_SPLITS"] = str(splits)
        try:
            ctxs.append(wdc.Context(cfg, max_batch=2, allocate_weights=not ctxs))
        finally:
            del os.environ["WDC_ATTN_SPLITS"]
    split, whole = ctxs
    W = synth.gen_weights(cfg)
    split.load_weights(W)
    whole.bind_weights(split.weights)
    host, dev = inputs(split, cfg, 2)
    zs = [d["z_T"] for d in dev]
    conds = [d["cond"] for d in dev]
    a = split.forward_batch(zs, 0.7, conds)
    b = whole.forward_batch(zs, 0.7, conds)
    for i in range(2):
        diff = rel_l2(a[i].cpu().numpy(), b[i].cpu().numpy())
        print(f"sample {i}: split vs unsplit rel_l2 {diff:.2e}")
        assert torch.isfinite(a[i]).all() and diff <= 1e-2
    assert not all(torch.equal(a[i], b[i]) for i in range(2))      # the split ran
    ref = dit.dit_forward(W, cfg, host[1]["z_T"], 0.7, host[1].get("cond"))
    err = rel_l2(a[1].cpu().numpy(), ref)
    print(f"sample 1 vs oracle {err:.2e}")
    assert err <= TOL_BF16_FINAL
