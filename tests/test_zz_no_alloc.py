"""The allocation-free block forward (bc_dit_block_forward_noalloc) against
bc_dit_block_forward with a caller workspace, through the C ABI: the same
kernels on the same inputs, so the outputs must be identical.  Two calls in a
row per block kind, the second with a smaller input (the shared scratch then
holds the first call's intermediates), and a shape over the scratch limit is
rejected before anything runs."""
import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def _dit_weights(bc, cfg, P):
    from paper_2608_28670_amd import loader
    dP = loader.upload(P, cfg)
    return dP, loader.block_list(cfg, dP)[0]


def _pair(bc, desc, w, x, c, x_txt=None):
    """(caller-workspace result, allocation-free result) on copies of x."""
    ws = torch.empty(bc.block_workspace_size(desc), dtype=torch.uint8, device=DEV)
    xa, xb = _f32(x), _f32(x)
    ta = _f32(x_txt) if x_txt is not None else None
    tb = _f32(x_txt) if x_txt is not None else None
    bc.dit_block_forward(desc, w, xa, _f32(c), ws, x_txt=ta)
    bc.dit_block_forward_noalloc(desc, w, xb, _f32(c), x_txt=tb)
    torch.cuda.synchronize()
    return (xa, ta), (xb, tb)


def test_noalloc_dit_block_two_calls(bclib):
    cfg = synth.scaled(synth.CONFIGS["dit_xl2"], depth=1)
    P = synth.params(cfg, names=[n for n, _ in synth.param_shapes(cfg) if n.startswith("blocks.0.")])
    dP, w = _dit_weights(bclib, cfg, P)
    for B in (16, 3):     # the bench's batch first, then a smaller one
        desc = bclib.block_desc(bclib.BLOCK_DIT, B, cfg.tokens, cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp,
                                bclib.BF16)
        assert bclib.block_workspace_size(desc) <= bclib.noalloc_scratch_bytes()
        x = synth.normal(f"noalloc/x{B}", (B, cfg.tokens, cfg.hidden))
        c = synth.normal(f"noalloc/c{B}", (B, cfg.hidden), 0.5)
        (ref, _), (got, _) = _pair(bclib, desc, w, x, c)
        assert torch.equal(ref, got), B
        upd = float(torch.linalg.vector_norm(got - _f32(x))) / float(torch.linalg.vector_norm(ref - _f32(x)))
        assert abs(upd - 1.0) < 1e-6
        print(f"noalloc DiT block B={B}: identical to the caller-workspace call", flush=True)


def test_noalloc_dual_block_two_calls(bclib):
    from paper_2608_28670_amd import loader
    cfg = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=256, heads=2, head_dim=128,
                       mlp=1024, latent=(16, 3, 20, 20), txt_tokens=40)
    P = synth.params(cfg, names=[n for n, _ in synth.param_shapes(cfg) if n.startswith("dual.0.")])
    dP = loader.upload(P, cfg)
    w = bclib.block_weights(loader._stream(dP, "dual.0.img."), loader._stream(dP, "dual.0.txt."))
    for B in (2, 1):
        desc = bclib.block_desc(bclib.BLOCK_DUAL, B, cfg.tokens, cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp,
                                bclib.BF16, T_txt=cfg.txt_tokens, rope=loader.rope_grid(cfg))
        x = synth.normal(f"noalloc/dx{B}", (B, cfg.tokens, cfg.hidden))
        xt = synth.normal(f"noalloc/dxt{B}", (B, cfg.txt_tokens, cfg.hidden))
        c = synth.normal(f"noalloc/dc{B}", (B, cfg.hidden), 0.5)
        (ra, rt), (ga, gt) = _pair(bclib, desc, w, x, c, x_txt=xt)
        assert torch.equal(ra, ga) and torch.equal(rt, gt), B


def test_noalloc_rejects_shape_over_the_limit(bclib):
    cfg = synth.CONFIGS["pixart"]
    # 16 samples of 4096 tokens need far more than the scratch holds
    desc = bclib.block_desc(bclib.BLOCK_DIT, 16, cfg.tokens, cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp, bclib.BF16)
    assert bclib.block_workspace_size(desc) > bclib.noalloc_scratch_bytes()
    x = torch.zeros((16, cfg.tokens, cfg.hidden), dtype=torch.float32, device=DEV)
    c = torch.zeros((16, cfg.hidden), dtype=torch.float32, device=DEV)
    w = bclib.block_weights({})
    with pytest.raises(bclib.BCError) as e:
        bclib.dit_block_forward_noalloc(desc, w, x, c)
    assert e.value.code == bclib.ERR_INVALID_ARG
    assert torch.count_nonzero(x) == 0
