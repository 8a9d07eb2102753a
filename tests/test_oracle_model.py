"""Pins for the oracle's denoiser, samplers and sampling loop.

The paper prints no activations or weights, so the blocks are pinned by
special cases (zero gates give the identity, one key gives attention = V,
token-permutation equivariance), by an independent fp64 re-expression built
from PyTorch CPU library routines (layer_norm, scaled_dot_product_attention,
gelu, linear), and by closed forms of the samplers.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import bary, model as om, sampler as osm



def tiny(**kw):
    return synth.scaled(synth.CONFIGS["tiny"], **kw)


def _torch_dit_block(P, pre, x, mod, heads):
    """DiT block from PyTorch library routines, fp64 on the CPU."""
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    x = t(x)
    s1, c1, g1, s2, c2, g2 = (t(m)[:, None, :] for m in mod)
    B, T, D = x.shape
    h = F.layer_norm(x, (D,), eps=1e-6) * (1 + c1) + s1
    qkv = F.linear(h, t(P[pre + "w_qkv"]), t(P[pre + "b_qkv"]))
    q, k, v = qkv.split(D, dim=-1)
    sh = lambda z: z.reshape(B, T, heads, D // heads).transpose(1, 2)
    a = F.scaled_dot_product_attention(sh(q), sh(k), sh(v)).transpose(1, 2).reshape(B, T, D)
    x = x + g1 * F.linear(a, t(P[pre + "w_o"]), t(P[pre + "b_o"]))
    h = F.layer_norm(x, (D,), eps=1e-6) * (1 + c2) + s2
    m = F.gelu(F.linear(h, t(P[pre + "w_fc1"]), t(P[pre + "b_fc1"])), approximate="tanh")
    return (x + g2 * F.linear(m, t(P[pre + "w_fc2"]), t(P[pre + "b_fc2"]))).numpy()


def test_dit_block_matches_torch_library_expression():
    cfg = tiny()
    P = synth.params(cfg)
    M = om.Model(cfg, P)
    g = np.random.default_rng(0)
    x = g.normal(size=(2, cfg.tokens, cfg.hidden))
    cond = M.condition(437.0, 2)
    mod = M.block_mod(1, cond)
    got = M.dit_block(1, x, mod)
    exp = _torch_dit_block(P, "blocks.1.", x, mod, cfg.heads)
    np.testing.assert_allclose(got, exp, rtol=1e-11, atol=1e-12)
    assert np.abs(got - x).max() > 1e-4          # the block is not the identity


def test_zero_gates_give_identity():
    cfg = tiny()
    P = synth.params(cfg)
    M = om.Model(cfg, P)
    x = np.random.default_rng(1).normal(size=(2, cfg.tokens, cfg.hidden))
    mod = M.block_mod(0, M.condition(10.0, 2))
    mod[2] = np.zeros_like(mod[2])
    mod[5] = np.zeros_like(mod[5])
    assert np.array_equal(M.dit_block(0, x, mod), x)


def test_attention_single_key_returns_value():
    g = np.random.default_rng(2)
    q = g.normal(size=(2, 3, 5, 8))
    k = g.normal(size=(2, 3, 1, 8))
    v = g.normal(size=(2, 3, 1, 8))
    np.testing.assert_allclose(om.attention(q, k, v), np.broadcast_to(v, (2, 3, 5, 8)), rtol=1e-15)


def test_attention_matches_torch_sdpa():
    g = np.random.default_rng(3)
    q, k, v = (g.normal(size=(2, 3, 17, 8)) for _ in range(3))
    exp = F.scaled_dot_product_attention(*(torch.from_numpy(a) for a in (q, k, v))).numpy()
    np.testing.assert_allclose(om.attention(q, k, v), exp, rtol=1e-12, atol=1e-13)


def test_block_is_token_permutation_equivariant():
    cfg = tiny()
    M = om.Model(cfg, synth.params(cfg))
    g = np.random.default_rng(4)
    x = g.normal(size=(2, cfg.tokens, cfg.hidden))
    perm = g.permutation(cfg.tokens)
    mod = M.block_mod(0, M.condition(500.0, 2))
    np.testing.assert_allclose(M.dit_block(0, x[:, perm], mod), M.dit_block(0, x, mod)[:, perm],
                               rtol=1e-12, atol=1e-13)


def test_elementwise_pieces_match_torch():
    z = np.linspace(-6, 6, 101)
    tz = torch.from_numpy(z)
    np.testing.assert_allclose(om.gelu_tanh(z), F.gelu(tz, approximate="tanh").numpy(), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(om.silu(z), F.silu(tz).numpy(), rtol=1e-14, atol=1e-15)
    x = np.random.default_rng(5).normal(size=(3, 40))
    np.testing.assert_allclose(om.layer_norm(x), F.layer_norm(torch.from_numpy(x), (40,), eps=1e-6).numpy(),
                               rtol=1e-12, atol=1e-13)


def test_timestep_embedding_special_values():
    e = om.timestep_embedding(0.0, 256)
    assert np.array_equal(e[0, :128], np.ones(128)) and np.array_equal(e[0, 128:], np.zeros(128))
    e = om.timestep_embedding(1.0, 256)
    assert abs(e[0, 0] - math.cos(1.0)) < 1e-15 and abs(e[0, 128] - math.sin(1.0)) < 1e-15
    # lowest frequency: 10000^(-127/128)
    assert abs(e[0, 255] - math.sin(10000.0 ** (-127 / 128))) < 1e-15


@pytest.mark.parametrize("shape,p", [((2, 3, 4, 6), 2), ((1, 2, 3, 4, 6), 2), ((2, 4, 8, 8), 1)])
def test_patchify_roundtrip_and_index_map(shape, p):
    lat = np.arange(np.prod(shape), dtype=np.float64).reshape(shape)
    tok = om.patchify(lat, p)
    back = om.unpatchify(tok, p, shape[1:], shape[1])
    assert np.array_equal(back, lat)
    if len(shape) == 4:
        B, C, H, W = shape
        b, i, j, ph, pw, c = B - 1, H // p - 1, 0, p - 1, 0, C - 1
        assert tok[b, i * (W // p) + j, (ph * p + pw) * C + c] == lat[b, c, i * p + ph, j * p + pw]


def test_final_layer_shape_and_linear_in_feature_after_norm():
    cfg = tiny()
    M = om.Model(cfg, synth.params(cfg))
    feat = np.random.default_rng(6).normal(size=(2, cfg.tokens, cfg.hidden))
    cond = M.condition(3.0, 2)
    out = M.final(feat, cond)
    assert out.shape == (2, cfg.out_ch) + cfg.latent[1:]
    # LayerNorm makes the final layer invariant to a positive rescale and shift of each token.
    np.testing.assert_allclose(M.final(3.0 * feat + 0.5, cond), out, rtol=0, atol=1e-6)  # eps=1e-6 inside the norm


# ---------------------------------------------------------------------------
# samplers
# ---------------------------------------------------------------------------

def test_alpha_bar_table_endpoints():
    ab = osm.alpha_bar_table()
    assert ab[0] == 1 - 1e-4
    # commonly quoted terminal value of the linear 1e-4..0.02 schedule over 1000 steps
    assert abs(ab[999] - 4.0358e-5) < 1e-9
    assert np.all(np.diff(ab) < 0)


def test_trailing_timesteps():
    assert list(osm.timesteps(10)) == [999, 899, 799, 699, 599, 499, 399, 299, 199, 99]
    t50 = osm.timesteps(50)
    assert t50[0] == 999 and t50[-1] == 19 and np.all(np.diff(t50) == -20)


def _consistent_eps_model(smp, x0):
    """Noise prediction consistent with a fixed clean sample x0."""
    def out(k, x):
        a = smp._a(k)
        return (x - math.sqrt(a) * x0) / math.sqrt(1 - a)
    return out


@pytest.mark.parametrize("kind", ["ddim", "dpmpp2m"])
def test_sampler_recovers_clean_sample_from_consistent_eps(kind):
    g = np.random.default_rng(7)
    x0 = g.normal(size=(2, 4, 3, 3))
    S = 20
    smp = osm.Sampler(kind, S, 4)
    x = g.normal(size=x0.shape)
    f = _consistent_eps_model(smp, x0)
    for k in range(S):
        x = smp.step(k, x, f(k, x))
    np.testing.assert_allclose(x, x0, rtol=1e-9, atol=1e-9)


def test_ddim_zero_eps_scales_latent():
    smp = osm.Sampler("ddim", 10, 4)
    x = np.ones((1, 4, 2, 2))
    y = smp.step(2, x, np.zeros_like(x))
    assert np.allclose(y, math.sqrt(smp._a(3) / smp._a(2)) * x, rtol=1e-14)


def test_dpmpp_first_step_equals_ddim():
    """First-order DPM-Solver++ is DDIM (a published identity)."""
    g = np.random.default_rng(8)
    x, eps = g.normal(size=(2, 4, 3, 3)), g.normal(size=(2, 4, 3, 3))
    a = osm.Sampler("ddim", 20, 4).step(0, x, eps)
    b = osm.Sampler("dpmpp2m", 20, 4).step(0, x, eps)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shift", [1.0, 7.0])
def test_euler_constant_velocity(shift):
    # The steps telescope: sum_k (sigma_{k+1} - sigma_k) = sigma_S - sigma_0 = -1
    # for any shift, so a constant velocity v moves x by exactly -v.
    smp = osm.Sampler("euler", 50, 4, shift)
    x1 = np.full((1, 4, 2, 2), 3.0)
    v = np.full_like(x1, 0.75)
    x = x1
    for k in range(50):
        x = smp.step(k, x, v)
    np.testing.assert_allclose(x, x1 - v, rtol=1e-13)


def test_time_shift_closed_forms():
    assert osm.shifted_sigma(0.5, 7.0) == pytest.approx(3.5 / 4.0, rel=1e-15)   # 7 (1/2) / (1 + 6 (1/2))
    assert osm.shifted_sigma(0.0, 7.0) == 0.0 and osm.shifted_sigma(1.0, 7.0) == 1.0
    sig = np.linspace(0, 1, 101)
    np.testing.assert_array_equal(osm.shifted_sigma(sig, 1.0), sig)
    sh = osm.shifted_sigma(sig, 7.0)
    assert np.all(np.diff(sh) > 0) and np.all(sh[1:-1] > sig[1:-1])          # increasing, above the diagonal
    # the inverse map is the shift by 1/s
    np.testing.assert_allclose(osm.shifted_sigma(sh, 1.0 / 7.0), sig, rtol=1e-13, atol=1e-15)
    # model times: 1000 sigma'(k) with sigma = 1 - k/S
    tm = osm.model_time("euler", 4, 7.0)
    np.testing.assert_allclose(tm, [1000.0, 1000.0 * 7 * 0.75 / (1 + 6 * 0.75), 1000.0 * 3.5 / 4.0,
                                    1000.0 * 7 * 0.25 / (1 + 6 * 0.25)], rtol=1e-15)


# ---------------------------------------------------------------------------
# the loop
# ---------------------------------------------------------------------------

class _LinearFeatureModel(om.Model):
    """Stand-in denoiser whose stepwise feature is an affine function of the
    model time, so a K=2 trapezoid forecast at delta = 1 must reproduce it."""

    def __init__(self, cfg):
        super().__init__(cfg, {})

    def condition(self, tau, B, labels=None, text=None):
        return {"c": tau}

    def embed(self, lat):
        return None

    def stack(self, x, cond, ctx):
        return np.full((1, 2, 3), 0.25 + 0.001 * cond["c"])

    def final(self, feat, cond):
        return np.zeros((1, 4, 2, 2)) + feat.mean()


def test_loop_forecasts_affine_feature_exactly():
    cfg = tiny(steps=20, interval=3, K=2)
    M = _LinearFeatureModel(cfg)
    mask = bary.make_mask(20, 3)
    tr = {}
    osm.sample(M, np.zeros((1, 4, 2, 2)), mask, 2, trace=tr)
    tin = osm.model_time("ddim", 20)
    for k in range(20):
        # step index is the node coordinate and tau is affine in k, so the feature is
        # affine in k; before the second full step a single node is copied
        exp = 0.25 + 0.001 * tin[0 if k < 3 else k]
        np.testing.assert_allclose(tr["feat"][k], exp, rtol=1e-10)   # eta-limited


def test_loop_all_full_mask_equals_vanilla():
    cfg = tiny(steps=4)
    M = om.Model(cfg, synth.params(cfg))
    xT = synth.latents(cfg).astype(np.float64)
    got = osm.sample(M, xT, np.ones(4, np.uint8), cfg.K)
    x = xT
    smp = osm.Sampler("ddim", 4, cfg.in_ch)
    tin = osm.model_time("ddim", 4)
    for k in range(4):
        cond = M.condition(tin[k], 2)
        x = smp.step(k, x, M.final(M.stack(M.embed(x), cond, None), cond))
    np.testing.assert_allclose(got, x, rtol=1e-13, atol=1e-15)


def test_loop_k1_forecast_reuses_last_feature():
    cfg = tiny(steps=6, K=1)
    M = om.Model(cfg, synth.params(cfg))
    tr = {}
    mask = np.array([1, 0, 0, 1, 0, 1], np.uint8)
    osm.sample(M, synth.latents(cfg).astype(np.float64), mask, 1, trace=tr)
    assert np.array_equal(tr["feat"][1], tr["feat"][0]) and np.array_equal(tr["feat"][4], tr["feat"][3])


def test_pixart_and_mmdit_shapes_run():
    pc = synth.scaled(synth.CONFIGS["pixart"], depth=1, hidden=64, heads=2, head_dim=32, mlp=128,
                      latent=(4, 8, 8), batch=1, ctx_tokens=5, ctx_dim=16)
    M = om.Model(pc, synth.params(pc))
    txt = synth.text(pc)
    x = osm.sample(M, synth.latents(pc).astype(np.float64), bary.make_mask(20, 4), 4, text=txt)
    assert x.shape == (1, 4, 8, 8) and np.all(np.isfinite(x))
    hc = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=64, heads=2, head_dim=32,
                      mlp=128, latent=(16, 2, 4, 6), txt_tokens=3)
    M = om.Model(hc, synth.params(hc))
    x = osm.sample(M, synth.latents(hc).astype(np.float64), bary.make_mask(6, 5), 3, text=synth.text(hc))
    assert x.shape == (1, 16, 2, 4, 6) and np.all(np.isfinite(x))


def test_bf16_rounding_matches_torch():
    a = synth.normal("probe", (1000,), 3.0)
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(synth.bf16_round(a), ref)


# ---------------------------------------------------------------------------
# classifier-free guidance (Sec. 4.1: the class-to-image runs use scale 1.5)
# ---------------------------------------------------------------------------

def _cond_tiny(**kw):
    return synth.scaled(synth.CONFIGS["tiny"], n_classes=10, **kw)


def _cfg_run(cfg, s, labels, mask):
    M = om.Model(cfg, synth.params(cfg))
    xT = synth.latents(cfg).astype(np.float64)
    return osm.sample(M, xT, mask, cfg.K, labels=labels, cfg_scale=s)


def test_cfg_scale_one_is_the_conditional_run_and_zero_the_null_class():
    cfg = _cond_tiny(steps=6)
    mask = bary.make_mask(6, 3)
    labels = np.array([3, 7])
    cond = _cfg_run(cfg, None, labels, mask)
    null = _cfg_run(cfg, None, np.full(2, cfg.n_classes), mask)
    np.testing.assert_allclose(_cfg_run(cfg, 1.0, labels, mask), cond, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(_cfg_run(cfg, 0.0, labels, mask), null, rtol=1e-12, atol=1e-14)
    assert not np.allclose(cond, null)


def test_cfg_one_step_is_affine_in_the_scale():
    # one DDIM step is affine in the model output, and the guided output is
    # affine in s: x(s) = x(0) + s (x(1) - x(0))
    cfg = _cond_tiny(steps=1)
    mask = np.ones(1, np.uint8)
    labels = np.array([1, 9])
    x0, x1, x15 = (_cfg_run(cfg, s, labels, mask) for s in (0.0, 1.0, 1.5))
    np.testing.assert_allclose(x15, x0 + 1.5 * (x1 - x0), rtol=1e-11, atol=1e-13)


def test_cfg_caches_both_halves():
    cfg = _cond_tiny(steps=6)
    M = om.Model(cfg, synth.params(cfg))
    tr = {}
    osm.sample(M, synth.latents(cfg).astype(np.float64), bary.make_mask(6, 3), cfg.K,
               labels=np.array([0, 5]), cfg_scale=1.5, trace=tr)
    assert tr["feat"][1].shape[0] == 4 and tr["out"][1].shape[0] == 2


# ---------------------------------------------------------------------------
# outputs at sampled query rows (used for full-size parity)
# ---------------------------------------------------------------------------

def test_block_rows_equal_rows_of_the_full_output():
    """`rows=` computes the same outputs as the whole block at those rows."""
    cfg = tiny()
    M = om.Model(cfg, synth.params(cfg))
    x = np.random.default_rng(12).normal(size=(2, cfg.tokens, cfg.hidden))
    mod = M.block_mod(0, M.condition(321.0, 2))
    rows = [0, 5, 17, cfg.tokens - 1]
    np.testing.assert_allclose(M.dit_block(0, x, mod, rows=rows), M.dit_block(0, x, mod)[:, rows],
                               rtol=1e-12, atol=1e-14)
    pc = synth.scaled(synth.CONFIGS["pixart"], depth=1, hidden=64, heads=2, head_dim=32, mlp=128,
                      latent=(4, 8, 8), batch=2, ctx_tokens=5, ctx_dim=16)
    Mp = om.Model(pc, synth.params(pc))
    ctx = Mp.context(synth.text(pc))
    xp = np.random.default_rng(13).normal(size=(2, pc.tokens, pc.hidden))
    cond = Mp.condition(40.0, 2)
    np.testing.assert_allclose(Mp.dit_block(0, xp, Mp.block_mod(0, cond), ctx, rows=[3, 9]),
                               Mp.dit_block(0, xp, Mp.block_mod(0, cond), ctx)[:, [3, 9]], rtol=1e-12, atol=1e-14)
    hc = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=64, heads=2, head_dim=32,
                      mlp=128, latent=(16, 2, 4, 6), txt_tokens=3)
    Mh = om.Model(hc, synth.params(hc))
    g = np.random.default_rng(14)
    xi, xt = g.normal(size=(2, hc.tokens, 64)), g.normal(size=(2, 3, 64))
    c = {"c": g.normal(size=(2, 64))}
    fi, ft = Mh.dual_block(0, xi, xt, c)
    ri, rt = Mh.dual_block(0, xi, xt, c, rows=([1, 11], [0, 2]))
    np.testing.assert_allclose(ri, fi[:, [1, 11]], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(rt, ft[:, [0, 2]], rtol=1e-12, atol=1e-14)
    z = np.concatenate([xi, xt], axis=1)
    np.testing.assert_allclose(Mh.single_block(0, z, c, hc.tokens, rows=[0, 7, hc.tokens + 1]),
                               Mh.single_block(0, z, c, hc.tokens)[:, [0, 7, hc.tokens + 1]], rtol=1e-12, atol=1e-14)
