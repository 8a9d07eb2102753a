"""GPU parity at the workloads' full sizes, through the C ABI.

* The video model's dual-stream and single-stream blocks at their real width
  (hidden 3072, 24 heads of 128, MLP 12288; the single-stream block's fused
  [qkv | mlp] projection is 21 504 wide and its output projection reads
  15 360) over the full 14 310 image + 256 text tokens, with QK RMSNorm and the
  3D rotary embedding.  The oracle (fp32) computes every key and value and the
  outputs of sampled query rows (`rows=`); the gate is relative L2 <= 2e-2 on
  those rows' outputs and on their updates (output - input).
* The PixArt block at the bench's batch of 4 x 4096 tokens (the attention
  kernel picks its query tile from the grid size), sampled rows per sample.
* The whole sampling loop of the video workload at real width and full token
  count (one dual and one single block, 50 shift-7 Euler steps, K = 3), its
  final latent compared at 4096 positions with the oracle's, stored by
  tests/golden/make_video_e2e.py (oracle only).
* The forecast microbenchmark [8, 16384, 3072] for every K in {2, 3, 4, 5} and
  both dtypes, on 20 000 sampled elements (componentwise error <= 1e-5
  relative to sum_j |w_j x_j| for fp32, one bf16 ulp of the exact value for
  bf16).
"""
import os

import numpy as np
import pytest

import synth
from oracle import bary, model as om

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.fullsize]
DEV = "cuda:0"
HERE = os.path.dirname(os.path.abspath(__file__))


def rel_l2(g, r):
    g, r = np.asarray(g, np.float64), np.asarray(r, np.float64)
    return float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30))


def _f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def _check(tag, got, x, exp, tol=2e-2):
    e_out, e_upd = rel_l2(got, exp), rel_l2(got - x, exp - x)
    print(f"{tag}: rel-L2 out {e_out:.2e} update {e_upd:.2e}", flush=True)
    assert e_out <= tol and e_upd <= tol, (tag, e_out, e_upd)


def _rows(n, k, seed):
    """k sampled token rows of n, always with the first and the last."""
    r = np.random.default_rng(seed).choice(np.arange(1, n - 1), k - 2, replace=False)
    return sorted({0, n - 1, *map(int, r)})


# ---------------------------------------------------------------------------
# the video model's blocks at real width
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def video():
    cfg = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, batch=1)
    assert (cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp, cfg.tokens, cfg.txt_tokens) == \
        (3072, 24, 128, 12288, 14310, 256)
    names = [n for n, _ in synth.param_shapes(cfg) if n.startswith(("dual.0.", "single.0."))]
    P = synth.params(cfg, names=names)
    return cfg, P


def _video_block(bc, cfg, P, kind, x, c, x_txt=None):
    from paper_2608_28670_amd import loader
    dP = loader.upload(P, cfg)
    if kind == bc.BLOCK_DUAL:
        w = bc.block_weights(loader._stream(dP, "dual.0.img."), loader._stream(dP, "dual.0.txt."))
    else:
        pre = "single.0."
        w = bc.block_weights({"w_mod": dP[pre + "w_mod"], "b_mod": dP[pre + "b_mod"], "w_qkv": dP[pre + "w_1"],
                              "b_qkv": dP[pre + "b_1"], "w_o": dP[pre + "w_2"], "b_o": dP[pre + "b_2"],
                              "q_norm": dP[pre + "q_norm"], "k_norm": dP[pre + "k_norm"]})
    desc = bc.block_desc(kind, 1, cfg.tokens, cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp, bc.BF16,
                         T_txt=cfg.txt_tokens, rope=loader.rope_grid(cfg))
    ws = torch.empty(bc.block_workspace_size(desc), dtype=torch.uint8, device=DEV)
    tx = _f32(x)
    tt = _f32(x_txt) if x_txt is not None else None
    bc.dit_block_forward(desc, w, tx, _f32(c), ws, x_txt=tt)
    torch.cuda.synchronize()
    out = tx.cpu().numpy(), (tt.cpu().numpy() if tt is not None else None)
    del dP, ws, tx, tt
    torch.cuda.empty_cache()
    return out


def test_dual_block_video_real_width(bclib, video):
    cfg, P = video
    M = om.Model(cfg, P, dtype=np.float32)
    x = synth.normal("vblk/x", (1, cfg.tokens, cfg.hidden))
    xt = synth.normal("vblk/xt", (1, cfg.txt_tokens, cfg.hidden))
    c = synth.normal("vblk/c", (1, cfg.hidden), 0.5)
    print("dual block 3072 x 24x128, 14310 + 256 tokens: GPU", flush=True)
    gi, gt = _video_block(bclib, cfg, P, bclib.BLOCK_DUAL, x, c, x_txt=xt)
    ri, rt = _rows(cfg.tokens, 48, 1), _rows(cfg.txt_tokens, 16, 2)
    print("dual block: oracle on sampled rows", flush=True)
    ei, et = M.dual_block(0, x, xt, {"c": c}, rows=(ri, rt))
    _check("dual block image rows", gi[:, ri], x[:, ri], ei)
    _check("dual block text rows", gt[:, rt], xt[:, rt], et)


def test_dual_block_video_real_width_ragged_text(bclib, video):
    """77 text tokens: the text stream's projections, which share launches with
    the image stream's, run one ragged row tile."""
    cfg0, P = video
    cfg = synth.scaled(cfg0, txt_tokens=77)
    M = om.Model(cfg, P, dtype=np.float32)
    x = synth.normal("vblk/x", (1, cfg.tokens, cfg.hidden))
    xt = synth.normal("vblk/xt77", (1, cfg.txt_tokens, cfg.hidden))
    c = synth.normal("vblk/c", (1, cfg.hidden), 0.5)
    print("dual block 3072 x 24x128, 14310 + 77 tokens: GPU", flush=True)
    gi, gt = _video_block(bclib, cfg, P, bclib.BLOCK_DUAL, x, c, x_txt=xt)
    ri, rt = _rows(cfg.tokens, 32, 5), _rows(cfg.txt_tokens, 16, 6)
    print("dual block, 77 text tokens: oracle on sampled rows", flush=True)
    ei, et = M.dual_block(0, x, xt, {"c": c}, rows=(ri, rt))
    _check("dual block (77 text tokens) image rows", gi[:, ri], x[:, ri], ei)
    _check("dual block (77 text tokens) text rows", gt[:, rt], xt[:, rt], et)


def test_single_block_video_real_width(bclib, video):
    cfg, P = video
    M = om.Model(cfg, P, dtype=np.float32)
    L = cfg.tokens + cfg.txt_tokens
    x = synth.normal("vblk/xs", (1, L, cfg.hidden))
    c = synth.normal("vblk/cs", (1, cfg.hidden), 0.5)
    print("single block 3072 x 24x128, [qkv | mlp] 21504, out 15360, 14566 tokens: GPU", flush=True)
    got, _ = _video_block(bclib, cfg, P, bclib.BLOCK_SINGLE, x, c)
    rows = _rows(cfg.tokens, 48, 3) + [cfg.tokens + r for r in _rows(cfg.txt_tokens, 16, 4)]
    print("single block: oracle on sampled rows", flush=True)
    exp = M.single_block(0, x, {"c": c}, cfg.tokens, rows=rows)
    _check("single block sampled rows", got[:, rows], x[:, rows], exp)


# ---------------------------------------------------------------------------
# PixArt block at the bench's batch
# ---------------------------------------------------------------------------

def test_pixart_block_batch4_full_tokens(bclib):
    from paper_2608_28670_amd import loader
    cfg = synth.scaled(synth.CONFIGS["pixart"], depth=1)
    B, D = cfg.batch, cfg.hidden
    assert (B, cfg.tokens) == (4, 4096)
    P = synth.params(cfg, names=[n for n, _ in synth.param_shapes(cfg) if n.startswith("blocks.0.")])
    M = om.Model(cfg, P, dtype=np.float32)
    x = synth.normal("pb4/x", (B, cfg.tokens, D))
    t6 = synth.normal("pb4/t6", (B, 6 * D), 0.3)
    ctx = synth.bf16_round(synth.normal("pb4/ctx", (B, cfg.ctx_tokens, D)))
    dP = loader.upload(P, cfg)
    pre = "blocks.0."
    w = bclib.block_weights(loader._stream(dP, pre), None,
                            {k: dP[pre + k] for k in ("wx_q", "bx_q", "wx_kv", "bx_kv", "wx_o", "bx_o")})
    desc = bclib.block_desc(bclib.BLOCK_PIXART, B, cfg.tokens, D, cfg.heads, cfg.head_dim, cfg.mlp, bclib.BF16,
                            T_ctx=cfg.ctx_tokens)
    ws = torch.empty(bclib.block_workspace_size(desc), dtype=torch.uint8, device=DEV)
    tx = _f32(x)
    print("pixart block B 4 x 4096 tokens: GPU", flush=True)
    bclib.dit_block_forward(desc, w, tx, _f32(t6), ws,
                            ctx=torch.from_numpy(ctx).to(DEV).to(torch.bfloat16))
    torch.cuda.synchronize()
    got = tx.cpu().numpy()
    y = om.linear(ctx.astype(np.float32), M.P[pre + "wx_kv"], M.P[pre + "bx_kv"])
    kv = [(om.split_heads(y[..., :D], cfg.heads), om.split_heads(y[..., D:], cfg.heads))]
    rows = _rows(cfg.tokens, 64, 5)
    print("pixart block: oracle on sampled rows", flush=True)
    exp = M.dit_block(0, x, M.block_mod(0, {"t6": t6}), {"kv": kv}, rows=rows)
    for b in range(B):
        _check(f"pixart block sample {b}", got[b:b + 1, rows], x[b:b + 1, rows], exp[b:b + 1])


# ---------------------------------------------------------------------------
# the video workload's sampling loop at real width and full token count
# ---------------------------------------------------------------------------

def _golden_video():
    idx, val = [], []
    with open(os.path.join(HERE, "golden", "video_e2e_sampled.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            i, v = line.split()
            idx.append(int(i))
            val.append(float(v))
    return np.array(idx), np.array(val)


def test_sample_video_real_width_full_tokens(bclib, video):
    from paper_2608_28670_amd import loader
    cfg = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, batch=1)
    idx, exp = _golden_video()
    P = synth.params(cfg)
    dm = loader.DeviceModel(cfg, P)
    mask = bary.make_mask(cfg.steps, cfg.interval)
    assert int(mask.sum()) == 11
    xT = synth.latents(cfg)
    x = _f32(xT)
    text = torch.from_numpy(synth.text(cfg)).to(DEV).to(torch.bfloat16)
    print("video sampling loop, real width, 1 dual + 1 single block, 50 steps: GPU", flush=True)
    ring = dm.sample(x, mask, text=text)
    torch.cuda.synchronize()
    got = x.cpu().numpy().reshape(-1)
    assert np.all(np.isfinite(got))
    err = rel_l2(got[idx], exp)
    print(f"video sampling loop: final latent rel-L2 {err:.2e} at {len(idx)} positions", flush=True)
    assert err <= 2e-2
    cnt, head, tn, _ = ring.state()
    full = [k for k in range(cfg.steps) if mask[k]]
    assert cnt == 3 and list(tn) == [float(k) for k in full[::-1][:3]]


# ---------------------------------------------------------------------------
# forecast microbenchmark, every (K, dtype)
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def c4_features():
    """Five [8, 16384, 3072] fp32 feature tensors; the K-node cases use the
    first K (the draws of slot j do not depend on K), bf16 cases their RNE
    rounding."""
    return synth.forecast_features(5, synth.FORECAST_SHAPE)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("K", [2, 3, 4, 5])
def test_forecast_full_size_every_k(bclib, c4_features, K, dt):
    shape = synth.FORECAST_SHAPE
    n = int(np.prod(shape))
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    s, t = synth.forecast_times(K)
    w = bary.bary_weights(s, t)
    storage = torch.empty((K, n), dtype=tdt, device=DEV)
    # node j (newest first) is pushed last-to-first, so it lands in slot K-1-j
    for j in range(K):
        storage[K - 1 - j].copy_(torch.from_numpy(c4_features[j].reshape(n)).to(DEV).to(tdt))
    ring = bclib.CacheRing(K, storage)
    for j in reversed(range(K)):
        ring.push(None, s[j])
    out = torch.empty(n, dtype=tdt, device=DEV)
    bclib.bary_extrapolate(ring, w, out)
    torch.cuda.synchronize()
    idx = np.concatenate([np.random.default_rng(K).integers(0, n, 20000), [0, n - 1]])
    nodes = [c4_features[j].reshape(n)[idx].astype(np.float64) for j in range(K)]
    if dt == "bf16":
        nodes = [synth.bf16_round(v.astype(np.float32)).astype(np.float64) for v in nodes]
    exact = sum(w[j] * nodes[j] for j in range(K))
    scale = sum(abs(w[j]) * np.abs(nodes[j]) for j in range(K))
    got = out[torch.from_numpy(idx).to(DEV)].float().cpu().numpy().astype(np.float64)
    if dt == "f32":
        err = float(np.max(np.abs(got - exact) / np.maximum(scale, 1e-30)))
        print(f"forecast K={K} f32: max componentwise rel err {err:.2e}", flush=True)
        assert err <= 1e-5
    else:
        ref = synth.bf16_round(exact.astype(np.float32)).astype(np.float64)
        # one bf16 ulp of the rounded exact value (the exact value is not
        # always representable in fp32, so compare in bf16 ulps of ref)
        ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 1e-38))) - 7)
        worst = float(np.max(np.abs(got - ref) / ulp))
        print(f"forecast K={K} bf16: max error {worst:.2f} ulp", flush=True)
        assert worst <= 1.0
    del storage, out
    torch.cuda.empty_cache()
