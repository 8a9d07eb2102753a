"""Pins for the query/key processing of the video model's blocks (QK RMSNorm and
the 3D rotary embedding of the image tokens): RMSNorm against PyTorch's
rms_norm, the rotation against complex multiplication, the relative-position
property of rotary embeddings, closed forms at the origin and for the first
pair of each axis, and the dual/single-stream blocks against a PyTorch
re-expression that applies both to the image tokens only."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import model as om


def _t(a):
    return torch.from_numpy(np.asarray(a, dtype=np.float64))


def test_rms_norm_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((3, 5, 128)) * 3.0
    w = 1.0 + 0.1 * rng.standard_normal(128)
    ref = F.rms_norm(_t(x), (128,), weight=_t(w), eps=1e-6).numpy()
    np.testing.assert_allclose(om.rms_norm(x, w), ref, rtol=1e-13, atol=1e-13)


def test_rope_axes_split():
    assert om.rope_axes(128) == (16, 56, 56)
    assert om.rope_axes(32) == (4, 14, 14)
    assert sum(om.rope_axes(64)) == 64


def test_rope_matches_complex_multiplication():
    rng = np.random.default_rng(2)
    grid, hd = (2, 3, 4), 32
    T = 24
    x = rng.standard_normal((2, 3, T, hd))
    ang = om.rope_angles(grid, hd, 256.0)
    xc = torch.view_as_complex(_t(x).reshape(2, 3, T, hd // 2, 2).contiguous())
    rot = torch.polar(torch.ones_like(_t(ang)), _t(ang))
    ref = torch.view_as_real(xc * rot).reshape(2, 3, T, hd).numpy()
    np.testing.assert_allclose(om.apply_rope(x, ang), ref, rtol=1e-13, atol=1e-13)


def test_rope_closed_forms():
    grid, hd, theta = (3, 4, 5), 32, 256.0
    ang = om.rope_angles(grid, hd, theta)
    assert np.all(ang[0] == 0.0)                         # token (0, 0, 0): the identity
    tok = lambda f, h, w: (f * grid[1] + h) * grid[2] + w
    a = ang[tok(2, 3, 4)]
    # the first pair of each axis turns by the axis position (frequency 1)
    assert a[0] == 2.0 and a[4 // 2] == 3.0 and a[(4 + 14) // 2] == 4.0
    # the second pair of the frame axis (d = 4): theta^(-2/4)
    assert a[1] == pytest.approx(2.0 * theta ** -0.5, rel=1e-15)


def test_rope_depends_on_relative_position_only():
    rng = np.random.default_rng(3)
    grid, hd = (4, 5, 6), 64
    ang = om.rope_angles(grid, hd, 256.0)
    q, k = rng.standard_normal(hd), rng.standard_normal(hd)
    tok = lambda f, h, w: (f * grid[1] + h) * grid[2] + w
    rot = lambda v, t: om.apply_rope(v[None], ang[t:t + 1])[0]
    for (a, b) in [((0, 1, 2), (1, 3, 0)), ((2, 0, 4), (0, 2, 1))]:
        d0 = rot(q, tok(*a)) @ rot(k, tok(*b))
        sh = lambda p: tuple(c + 1 for c in p)
        d1 = rot(q, tok(*sh(a))) @ rot(k, tok(*sh(b)))
        assert d0 == pytest.approx(d1, rel=1e-12)
    # norms of the pairs are unchanged
    r = rot(q, tok(3, 4, 5))
    np.testing.assert_allclose(np.hypot(r[0::2], r[1::2]), np.hypot(q[0::2], q[1::2]), rtol=1e-13)


def _mm_cfg():
    return synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=64, heads=2, head_dim=32,
                        mlp=128, latent=(16, 2, 4, 6), txt_tokens=3, batch=2)


def _torch_qk(q, k, P, pre, n_img, ang):
    q = F.rms_norm(q, (q.shape[-1],), weight=_t(P[pre + "q_norm"]), eps=1e-6)
    k = F.rms_norm(k, (k.shape[-1],), weight=_t(P[pre + "k_norm"]), eps=1e-6)
    rot = torch.polar(torch.ones_like(_t(ang)), _t(ang))

    def r(z):
        if n_img == 0:
            return z
        B, H, T, hd = z.shape
        zi = torch.view_as_complex(z[:, :, :n_img].reshape(B, H, n_img, hd // 2, 2).contiguous())
        zi = torch.view_as_real(zi * rot).reshape(B, H, n_img, hd)
        return torch.cat([zi, z[:, :, n_img:]], dim=2)
    return r(q), r(k)


def test_dual_block_against_torch():
    cfg = _mm_cfg()
    assert cfg.qk_norm and cfg.rope_theta == 256.0
    P = synth.params(cfg)
    M = om.Model(cfg, P)
    B, D, H, hd = 2, cfg.hidden, cfg.heads, cfg.head_dim
    rng = np.random.default_rng(4)
    xi, xt = rng.standard_normal((B, cfg.tokens, D)), rng.standard_normal((B, cfg.txt_tokens, D))
    c = rng.standard_normal((B, D)) * 0.5
    gi, gt = M.dual_block(0, xi, xt, {"c": c})
    ang = om.rope_angles(M.token_grid(), hd, cfg.rope_theta)
    Ti = cfg.tokens
    qs, ks, vs, mods = [], [], [], {}
    for s, x in (("img", xi), ("txt", xt)):
        pre = f"dual.0.{s}."
        m = F.linear(F.silu(_t(c)), _t(P[pre + "w_mod"]), _t(P[pre + "b_mod"]))
        mods[s] = m.split(D, dim=-1)
        h = F.layer_norm(_t(x), (D,), eps=1e-6) * (1 + mods[s][1][:, None]) + mods[s][0][:, None]
        qkv = F.linear(h, _t(P[pre + "w_qkv"]), _t(P[pre + "b_qkv"]))
        sh = lambda z: z.reshape(B, -1, H, hd).transpose(1, 2)
        q, k, v = (sh(z) for z in qkv.split(D, dim=-1))
        q, k = _torch_qk(q, k, P, pre, Ti if s == "img" else 0, ang)
        qs.append(q); ks.append(k); vs.append(v)
    a = F.scaled_dot_product_attention(torch.cat(qs, 2), torch.cat(ks, 2), torch.cat(vs, 2))
    a = a.transpose(1, 2).reshape(B, -1, D)
    outs = []
    for s, x, a_s in (("img", xi, a[:, :Ti]), ("txt", xt, a[:, Ti:])):
        pre = f"dual.0.{s}."
        s1, c1, g1, s2, c2, g2 = (z[:, None] for z in mods[s])
        y = _t(x) + g1 * F.linear(a_s, _t(P[pre + "w_o"]), _t(P[pre + "b_o"]))
        h = F.layer_norm(y, (D,), eps=1e-6) * (1 + c2) + s2
        mm = F.gelu(F.linear(h, _t(P[pre + "w_fc1"]), _t(P[pre + "b_fc1"])), approximate="tanh")
        outs.append((y + g2 * F.linear(mm, _t(P[pre + "w_fc2"]), _t(P[pre + "b_fc2"]))).numpy())
    np.testing.assert_allclose(gi, outs[0], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(gt, outs[1], rtol=1e-10, atol=1e-12)


def test_single_block_against_torch():
    cfg = _mm_cfg()
    P = synth.params(cfg)
    M = om.Model(cfg, P)
    B, D, H, hd, Fm = 2, cfg.hidden, cfg.heads, cfg.head_dim, cfg.mlp
    Ti, L = cfg.tokens, cfg.tokens + cfg.txt_tokens
    rng = np.random.default_rng(5)
    x = rng.standard_normal((B, L, D))
    c = rng.standard_normal((B, D)) * 0.5
    got = M.single_block(0, x, {"c": c}, Ti)
    pre = "single.0."
    m = F.linear(F.silu(_t(c)), _t(P[pre + "w_mod"]), _t(P[pre + "b_mod"]))
    s1, c1, g1 = (z[:, None] for z in m.split(D, dim=-1))
    h = F.layer_norm(_t(x), (D,), eps=1e-6) * (1 + c1) + s1
    y = F.linear(h, _t(P[pre + "w_1"]), _t(P[pre + "b_1"]))
    sh = lambda z: z.reshape(B, L, H, hd).transpose(1, 2)
    q, k, v = (sh(z) for z in y[..., :3 * D].split(D, dim=-1))
    q, k = _torch_qk(q, k, P, pre, Ti, om.rope_angles(M.token_grid(), hd, cfg.rope_theta))
    a = F.scaled_dot_product_attention(q, k, v).transpose(1, 2).reshape(B, L, D)
    z = torch.cat([a, F.gelu(y[..., 3 * D:], approximate="tanh")], dim=-1)
    ref = (_t(x) + g1 * F.linear(z, _t(P[pre + "w_2"]), _t(P[pre + "b_2"]))).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-12)
    # without the image-token count, no rotation: a different result
    assert not np.allclose(M.single_block(0, x, {"c": c}), got)
