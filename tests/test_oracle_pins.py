"""Independent pins for the parts of the oracle that the block-level pins do not
reach: the PixArt model's conditioning, caption context and cross-attention,
the final layer's adaLN of every model kind, and the second-order step of
DPM-Solver++(2M).

* Whole-model forward passes (embedding, conditioning, every block kind, the
  final layer and unpatchify) are re-expressed from PyTorch CPU library
  routines in fp64: `F.unfold`/`F.fold` for the patch maps, `F.linear`,
  `F.silu`, `F.gelu(approximate="tanh")`, `F.layer_norm`, `F.rms_norm` and
  `F.scaled_dot_product_attention` with Tq != Tk for the cross-attention, the
  keys and values split as a (2, heads, head_dim) view of the projection.
* Special cases: with one context token the cross-attention returns that
  token's value projection for every query, so its output is
  (ctx Wv^T + bv) Wo^T + bo whatever the queries are.
* DPM-Solver++(2M) (the published multistep solver in data-prediction form):
  when the data prediction is affine in lambda, the combined estimate D of a
  second-order step equals the prediction at the midpoint lambda_k + h_k / 2;
  its global error falls by 4x when the step count doubles (DDIM's by 2x),
  measured against the closed-form solution of the probability-flow ODE; and
  a two-step example worked by hand (`golden/dpmpp2m_worked.txt`).

Every pin is checked to fail under the mistake it is meant to catch, planted
in a patched copy of the oracle (swapped key/value halves, a dropped output
bias, a gated cross-attention, swapped shift and scale, an inverted step
ratio r, a flipped sign on 1/(2r)).
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import model as om, sampler as osm

HERE = os.path.dirname(os.path.abspath(__file__))


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


# ---------------------------------------------------------------------------
# whole-model forward from PyTorch library routines
# ---------------------------------------------------------------------------

def _torch_patchify(lat, p):
    """[B, C, H, W] -> [B, T, p*p*C], features in (p_h, p_w, c) order, via unfold
    (which lists a patch channel-major: c * p^2 + p_h * p + p_w)."""
    if lat.dim() == 5:   # video: frames folded into the batch, tokens frame-major
        B, C, Fr, H, W = lat.shape
        x = lat.permute(0, 2, 1, 3, 4).reshape(B * Fr, C, H, W)
        tok = _torch_patchify(x, p)
        return tok.reshape(B, Fr * tok.shape[1], tok.shape[2])
    B, C = lat.shape[:2]
    u = F.unfold(lat, kernel_size=p, stride=p)                 # [B, C p p, L]
    return u.reshape(B, C, p * p, -1).permute(0, 3, 2, 1).reshape(B, -1, p * p * C)


def _torch_unpatchify(tok, p, latent, C):
    if len(latent) == 4:
        _, Fr, H, W = latent
        B = tok.shape[0]
        x = _torch_unpatchify(tok.reshape(B * Fr, -1, tok.shape[2]), p, (C, H, W), C)
        return x.reshape(B, Fr, C, H, W).permute(0, 2, 1, 3, 4)
    _, H, W = latent
    B, L, _ = tok.shape
    u = tok.reshape(B, L, p * p, C).permute(0, 3, 2, 1).reshape(B, C * p * p, L)
    return F.fold(u, output_size=(H, W), kernel_size=p, stride=p)


def _torch_t_embed(P, tau, B, dim):
    half = dim // 2
    f = torch.exp(-math.log(10000.0) * torch.arange(half, dtype=torch.float64) / half)
    a = torch.full((B, 1), float(tau), dtype=torch.float64) * f[None]
    e = torch.cat([torch.cos(a), torch.sin(a)], dim=-1)
    return F.linear(F.silu(F.linear(e, _t(P["t_w1"]), _t(P["t_b1"]))), _t(P["t_w2"]), _t(P["t_b2"]))


def _ln_mod(x, shift, scale):
    D = x.shape[-1]
    return F.layer_norm(x, (D,), eps=1e-6) * (1 + scale[:, None]) + shift[:, None]


def _heads(z, H):
    B, T, D = z.shape
    return z.reshape(B, T, H, D // H).transpose(1, 2)


def _merge(z):
    B, H, T, d = z.shape
    return z.transpose(1, 2).reshape(B, T, H * d)


def _torch_qk(cfg, P, pre, q, k, n_img, grid):
    if cfg.qk_norm:
        q = F.rms_norm(q, (cfg.head_dim,), weight=_t(P[pre + "q_norm"]), eps=1e-6)
        k = F.rms_norm(k, (cfg.head_dim,), weight=_t(P[pre + "k_norm"]), eps=1e-6)
    if cfg.rope_theta and n_img:
        # complex rotation by angles built per axis: frequencies theta^(-2j/d)
        hd = cfg.head_dim
        axes = (hd // 8, (hd - hd // 8) // 2, hd - hd // 8 - (hd - hd // 8) // 2)
        pos = torch.stack(torch.meshgrid(*(torch.arange(n, dtype=torch.float64) for n in grid),
                                         indexing="ij"), -1).reshape(-1, 3)
        ang = torch.cat([pos[:, i:i + 1] * cfg.rope_theta ** (-torch.arange(0, d, 2, dtype=torch.float64) / d)
                         for i, d in enumerate(axes)], dim=1)
        rot = torch.polar(torch.ones_like(ang), ang)

        def r(z):
            B, H, T, _ = z.shape
            zi = torch.view_as_complex(z[:, :, :n_img].reshape(B, H, n_img, hd // 2, 2).contiguous())
            return torch.cat([torch.view_as_real(zi * rot).reshape(B, H, n_img, hd), z[:, :, n_img:]], dim=2)
        q, k = r(q), r(k)
    return q, k


def _torch_dit_like_block(cfg, P, pre, x, mod, ctx):
    """DiT block (and PixArt's, with its cross-attention after self-attention)."""
    D, H = cfg.hidden, cfg.heads
    s1, c1, g1, s2, c2, g2 = mod
    h = _ln_mod(x, s1, c1)
    q, k, v = (_heads(z, H) for z in F.linear(h, _t(P[pre + "w_qkv"]), _t(P[pre + "b_qkv"])).split(D, -1))
    x = x + g1[:, None] * F.linear(_merge(F.scaled_dot_product_attention(q, k, v)),
                                   _t(P[pre + "w_o"]), _t(P[pre + "b_o"]))
    if cfg.kind == "pixart":
        B, Tc, _ = ctx.shape
        kv = F.linear(ctx, _t(P[pre + "wx_kv"]), _t(P[pre + "bx_kv"])).reshape(B, Tc, 2, H, D // H)
        kx, vx = kv[:, :, 0].transpose(1, 2), kv[:, :, 1].transpose(1, 2)
        qx = _heads(F.linear(x, _t(P[pre + "wx_q"]), _t(P[pre + "bx_q"])), H)
        x = x + F.linear(_merge(F.scaled_dot_product_attention(qx, kx, vx)), _t(P[pre + "wx_o"]), _t(P[pre + "bx_o"]))
    h = _ln_mod(x, s2, c2)
    m = F.gelu(F.linear(h, _t(P[pre + "w_fc1"]), _t(P[pre + "b_fc1"])), approximate="tanh")
    return x + g2[:, None] * F.linear(m, _t(P[pre + "w_fc2"]), _t(P[pre + "b_fc2"]))


def torch_forward(cfg, P, lat, tau, labels=None, text=None):
    """Model output [B, C_out, ...] of one denoiser evaluation."""
    D, H, p = cfg.hidden, cfg.heads, cfg.p
    lat = _t(lat)
    B = lat.shape[0]
    x = F.linear(_torch_patchify(lat, p), _t(P["patch_w"]), _t(P["patch_b"])) + _t(P["pos"])[None]
    t = _torch_t_embed(P, tau, B, cfg.freq_dim)
    if cfg.kind == "dit":
        c = t + _t(P["y_table"])[torch.as_tensor(labels)] if cfg.n_classes else t
        for l in range(cfg.depth):
            pre = f"blocks.{l}."
            mod = F.linear(F.silu(c), _t(P[pre + "w_mod"]), _t(P[pre + "b_mod"])).chunk(6, dim=-1)
            x = _torch_dit_like_block(cfg, P, pre, x, mod, None)
        shift, scale = F.linear(F.silu(c), _t(P["final_w_mod"]), _t(P["final_b_mod"])).chunk(2, dim=-1)
    elif cfg.kind == "pixart":
        ctx = F.linear(F.gelu(F.linear(_t(text), _t(P["cap_w1"]), _t(P["cap_b1"])), approximate="tanh"),
                       _t(P["cap_w2"]), _t(P["cap_b2"]))
        t6 = F.linear(F.silu(t), _t(P["t6_w"]), _t(P["t6_b"]))
        for l in range(cfg.depth):
            pre = f"blocks.{l}."
            mod = (t6.reshape(B, 6, D) + _t(P[pre + "table"])[None]).unbind(1)
            x = _torch_dit_like_block(cfg, P, pre, x, mod, ctx)
        shift, scale = (_t(P["final_table"])[None] + t[:, None]).unbind(1)
    else:
        txt = _t(text)
        c = t + F.linear(txt.mean(dim=1), _t(P["txt_w"]), _t(P["txt_b"]))
        Ti = x.shape[1]
        grid = (cfg.latent[1], cfg.latent[2] // p, cfg.latent[3] // p)
        xt = txt
        for l in range(cfg.depth):
            st = {}
            for s, z in (("img", x), ("txt", xt)):
                pre = f"dual.{l}.{s}."
                mod = F.linear(F.silu(c), _t(P[pre + "w_mod"]), _t(P[pre + "b_mod"])).chunk(6, dim=-1)
                q, k, v = (_heads(y, H) for y in
                           F.linear(_ln_mod(z, mod[0], mod[1]), _t(P[pre + "w_qkv"]), _t(P[pre + "b_qkv"])).split(D, -1))
                q, k = _torch_qk(cfg, P, pre, q, k, Ti if s == "img" else 0, grid)
                st[s] = (z, mod, q, k, v)
            a = _merge(F.scaled_dot_product_attention(*(torch.cat([st["img"][i], st["txt"][i]], dim=2)
                                                        for i in (2, 3, 4))))
            outs = []
            for s, a_s in (("img", a[:, :Ti]), ("txt", a[:, Ti:])):
                pre = f"dual.{l}.{s}."
                z, mod = st[s][0], st[s][1]
                z = z + mod[2][:, None] * F.linear(a_s, _t(P[pre + "w_o"]), _t(P[pre + "b_o"]))
                m = F.gelu(F.linear(_ln_mod(z, mod[3], mod[4]), _t(P[pre + "w_fc1"]), _t(P[pre + "b_fc1"])),
                           approximate="tanh")
                outs.append(z + mod[5][:, None] * F.linear(m, _t(P[pre + "w_fc2"]), _t(P[pre + "b_fc2"])))
            x, xt = outs
        z = torch.cat([x, xt], dim=1)
        for l in range(cfg.depth_single):
            pre = f"single.{l}."
            s1, c1, g1 = F.linear(F.silu(c), _t(P[pre + "w_mod"]), _t(P[pre + "b_mod"])).chunk(3, dim=-1)
            y = F.linear(_ln_mod(z, s1, c1), _t(P[pre + "w_1"]), _t(P[pre + "b_1"]))
            q, k, v = (_heads(u, H) for u in y[..., :3 * D].split(D, -1))
            q, k = _torch_qk(cfg, P, pre, q, k, Ti, grid)
            a = _merge(F.scaled_dot_product_attention(q, k, v))
            z = z + g1[:, None] * F.linear(torch.cat([a, F.gelu(y[..., 3 * D:], approximate="tanh")], -1),
                                           _t(P[pre + "w_2"]), _t(P[pre + "b_2"]))
        x = z[:, :Ti]
        shift, scale = F.linear(F.silu(c), _t(P["final_w_mod"]), _t(P["final_b_mod"])).chunk(2, dim=-1)
    y = F.linear(_ln_mod(x, shift, scale), _t(P["final_w"]), _t(P["final_b"]))
    return _torch_unpatchify(y, p, cfg.latent, cfg.out_ch).numpy()


def oracle_forward(M, lat, tau, labels=None, text=None):
    cfg = M.cfg
    B = lat.shape[0]
    cond = M.condition(tau, B, labels, text)
    ctx = M.context(text) if cfg.kind != "dit" else None
    return M.final(M.stack(M.embed(lat), cond, ctx), cond)


def _pixart_cfg(**kw):
    base = dict(depth=2, hidden=64, heads=2, head_dim=32, mlp=128, latent=(4, 8, 8), batch=2,
                ctx_tokens=5, ctx_dim=48)
    base.update(kw)
    return synth.scaled(synth.CONFIGS["pixart"], **base)


def _cases():
    dit = synth.scaled(synth.CONFIGS["dit_xl2"], depth=2, hidden=64, heads=2, head_dim=32, mlp=128,
                       latent=(4, 8, 8), batch=2, n_classes=10, dtype="f32")
    pix = _pixart_cfg(dtype="f32")
    mm = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=64, heads=2, head_dim=32,
                      mlp=128, latent=(16, 2, 4, 6), txt_tokens=3, dtype="f32")
    return {"dit": dit, "pixart": pix, "mmdit": mm}


def _inputs(cfg):
    lat = synth.normal(f"pins/{cfg.name}/lat", (2,) + tuple(cfg.latent)).astype(np.float64)
    labels = np.array([3, 7]) if cfg.n_classes else None
    text = synth.text(cfg, batch=2).astype(np.float64) if cfg.kind != "dit" else None
    return lat, labels, text


def _forward_error(M, tau=613.0):
    cfg = M.cfg
    lat, labels, text = _inputs(cfg)
    got = oracle_forward(M, lat, tau, labels, text)
    exp = torch_forward(cfg, M.P, lat, tau, labels, text)
    assert got.shape == exp.shape == (2, cfg.out_ch) + tuple(cfg.latent[1:])
    return float(np.abs(got - exp).max() / np.abs(exp).max())


@pytest.mark.parametrize("kind", ["dit", "pixart", "mmdit"])
def test_model_forward_matches_torch_library_expression(kind):
    cfg = _cases()[kind]
    M = om.Model(cfg, synth.params(cfg))
    assert _forward_error(M) <= 1e-12


def test_torch_patch_maps_invert():
    for shape, p in (((2, 3, 4, 6), 2), ((1, 2, 3, 4, 6), 2)):
        lat = _t(np.arange(np.prod(shape), dtype=np.float64).reshape(shape))
        tok = _torch_patchify(lat, p)
        assert torch.equal(_torch_unpatchify(tok, p, shape[1:], shape[1]), lat)
        assert np.array_equal(tok.numpy(), om.patchify(lat.numpy(), p))


# ---------------------------------------------------------------------------
# PixArt cross-attention special cases
# ---------------------------------------------------------------------------

def _cross_only(M, l, x, ctx):
    """The block with both gates zero: x + cross-attention(x, ctx) alone."""
    mod = [np.zeros((x.shape[0], M.cfg.hidden)) for _ in range(6)]
    return M.dit_block(l, x, mod, ctx) - x


def _cross_single_token_error(M):
    cfg, P = M.cfg, M.P
    D = cfg.hidden
    text = synth.text(synth.scaled(cfg, ctx_tokens=1), batch=2).astype(np.float64)
    ctx = M.context(text)
    x = synth.normal("pins/pix/x1", (2, cfg.tokens, D)).astype(np.float64)
    got = _cross_only(M, 1, x, ctx)
    # one key: softmax weight 1, so every query returns the value row
    c = ctx["ctx"][:, 0]                                       # [B, D]
    v = c @ P["blocks.1.wx_kv"][D:].T + P["blocks.1.bx_kv"][D:]
    exp = (v @ P["blocks.1.wx_o"].T + P["blocks.1.bx_o"])[:, None, :]
    return float(np.abs(got - exp).max() / np.abs(exp).max())


def test_cross_attention_one_context_token_returns_value_projection():
    cfg = _pixart_cfg(ctx_tokens=1, dtype="f32")
    M = om.Model(cfg, synth.params(cfg))
    assert _cross_single_token_error(M) <= 1e-13


def test_cross_attention_ignores_context_order_and_query_weights_with_one_token():
    cfg = _pixart_cfg(dtype="f32")
    P = synth.params(cfg)
    M = om.Model(cfg, P)
    text = synth.text(cfg, batch=2).astype(np.float64)
    x = synth.normal("pins/pix/x2", (2, cfg.tokens, cfg.hidden)).astype(np.float64)
    base = _cross_only(M, 0, x, M.context(text))
    perm = np.random.default_rng(11).permutation(cfg.ctx_tokens)
    np.testing.assert_allclose(_cross_only(M, 0, x, M.context(text[:, perm])), base, rtol=1e-12, atol=1e-14)
    # with one context token the queries do not matter
    one = synth.scaled(cfg, ctx_tokens=1)
    P2 = dict(P)
    P2["blocks.0.wx_q"] = 3.0 * P["blocks.0.wx_q"] + 0.1
    t1 = text[:, :1]
    a = _cross_only(om.Model(one, P), 0, x, om.Model(one, P).context(t1))
    b = _cross_only(om.Model(one, P2), 0, x, om.Model(one, P2).context(t1))
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------------------
# planted mistakes: each pin above must fail on the oracle with the mistake
# ---------------------------------------------------------------------------

class _SwappedKV(om.Model):
    def context(self, text):
        out = super().context(text)
        if "kv" in out:
            out["kv"] = [(v, k) for k, v in out["kv"]]
        return out


class _GatedCross(om.Model):
    """Cross-attention scaled by the attention gate (a gate the PixArt block does not have)."""
    def dit_block(self, l, x, mod, ctx=None, modules=None):
        P, D, H = self.P, self.cfg.hidden, self.cfg.heads
        pre = f"blocks.{l}."
        s1, sc1, g1, s2, sc2, g2 = mod
        qkv = om.linear(om.modulate(om.layer_norm(x), s1, sc1), P[pre + "w_qkv"], P[pre + "b_qkv"])
        q, k, v = (om.split_heads(qkv[..., i * D:(i + 1) * D], H) for i in range(3))
        x = x + g1[:, None, :] * om.linear(om.merge_heads(om.attention(q, k, v)), P[pre + "w_o"], P[pre + "b_o"])
        kx, vx = ctx["kv"][l]
        qx = om.split_heads(om.linear(x, P[pre + "wx_q"], P[pre + "bx_q"]), H)
        x = x + g1[:, None, :] * om.linear(om.merge_heads(om.attention(qx, kx, vx)), P[pre + "wx_o"], P[pre + "bx_o"])
        m = om.gelu_tanh(om.linear(om.modulate(om.layer_norm(x), s2, sc2), P[pre + "w_fc1"], P[pre + "b_fc1"]))
        return x + g2[:, None, :] * om.linear(m, P[pre + "w_fc2"], P[pre + "b_fc2"])


class _SwappedFinalShiftScale(om.Model):
    def final(self, feat, cond):
        cfg, P = self.cfg, self.P
        D = cfg.hidden
        if cfg.kind == "pixart":
            shift = P["final_table"][1][None] + cond["t"]
            scale = P["final_table"][0][None] + cond["t"]
        else:
            m = om.linear(om.silu(cond["c"]), P["final_w_mod"], P["final_b_mod"])
            shift, scale = m[:, D:], m[:, :D]
        h = om.modulate(om.layer_norm(np.asarray(feat, dtype=self.dt)), shift, scale)
        return om.unpatchify(om.linear(h, P["final_w"], P["final_b"]), cfg.p, cfg.latent, cfg.out_ch)


class _TableOnlyModulation(om.Model):
    def block_mod(self, l, cond):
        if self.cfg.kind != "pixart":
            return super().block_mod(l, cond)
        D = self.cfg.hidden
        m = np.broadcast_to(self.P[f"blocks.{l}.table"].reshape(1, 6 * D), cond["t6"].shape)
        return [m[:, i * D:(i + 1) * D] for i in range(6)]


def test_planted_mistakes_fail_the_pins():
    cases = _cases()
    pix = cases["pixart"]
    Ppix = synth.params(pix)
    # swapped key/value halves of the context projection
    assert _forward_error(_SwappedKV(pix, Ppix)) > 1e-6
    one = _pixart_cfg(ctx_tokens=1, dtype="f32")
    P1 = synth.params(one)
    assert _cross_single_token_error(_SwappedKV(one, P1)) > 1e-3
    # dropped cross-attention output bias
    P_nob = dict(Ppix)
    P_nob["blocks.0.bx_o"] = np.zeros_like(Ppix["blocks.0.bx_o"])
    M = om.Model(pix, Ppix)
    lat, labels, text = _inputs(pix)
    exp = torch_forward(pix, Ppix, lat, 613.0, labels, text)
    got = oracle_forward(om.Model(pix, P_nob), lat, 613.0, labels, text)
    assert np.abs(got - exp).max() / np.abs(exp).max() > 1e-6
    P1b = dict(P1)
    P1b["blocks.1.bx_o"] = np.zeros_like(P1["blocks.1.bx_o"])
    assert _cross_single_token_error_against(om.Model(one, P1b), P1) > 1e-3
    # a gate on the cross-attention
    assert _forward_error(_GatedCross(pix, Ppix)) > 1e-6
    # t6 + table modulation reduced to the table
    assert _forward_error(_TableOnlyModulation(pix, Ppix)) > 1e-6
    # shift and scale of the final layer swapped, for every model kind
    for kind, cfg in cases.items():
        assert _forward_error(_SwappedFinalShiftScale(cfg, synth.params(cfg))) > 1e-6, kind
    assert _forward_error(M) <= 1e-12


def _cross_single_token_error_against(M, P_true):
    """As _cross_single_token_error, with the expected value from P_true."""
    cfg = M.cfg
    D = cfg.hidden
    text = synth.text(synth.scaled(cfg, ctx_tokens=1), batch=2).astype(np.float64)
    x = synth.normal("pins/pix/x1", (2, cfg.tokens, D)).astype(np.float64)
    got = _cross_only(M, 1, x, M.context(text))
    ctx = om.Model(cfg, P_true).context(text)["ctx"][:, 0]
    v = ctx @ P_true["blocks.1.wx_kv"][D:].T + P_true["blocks.1.bx_kv"][D:]
    exp = (v @ P_true["blocks.1.wx_o"].T + P_true["blocks.1.bx_o"])[:, None, :]
    return float(np.abs(got - exp).max() / np.abs(exp).max())


# ---------------------------------------------------------------------------
# DPM-Solver++(2M)
# ---------------------------------------------------------------------------

def _alpha_sigma_lambda(smp, k):
    a = smp._a(k)
    al, sg = math.sqrt(a), math.sqrt(1.0 - a)
    return al, sg, math.log(al / sg)


def _eps_for(smp, k, x, x0):
    """The noise prediction whose data prediction at step k is x0."""
    al, sg, _ = _alpha_sigma_lambda(smp, k)
    return (x - al * x0) / sg


class _SecondOrderVariant(osm.Sampler):
    """DPM-Solver++(2M) with a planted change in the combined estimate D."""
    def combine(self, x0, prev_x0, r):
        raise NotImplementedError

    def step(self, k, x, out):
        if self.kind != "dpmpp2m" or k == 0 or k == self.S - 1:
            return super().step(k, x, out)
        eps = out[:, :self.C]
        al, sg, lam = _alpha_sigma_lambda(self, k)
        al2, sg2, lam2 = _alpha_sigma_lambda(self, k + 1)
        x0 = (x - sg * eps) / al
        h = lam2 - lam
        d = self.combine(x0, self.prev_x0, self.prev_h / h)
        self.prev_x0, self.prev_h = x0, h
        return (sg2 / sg) * x - al2 * (math.exp(-h) - 1.0) * d


class _InvertedR(_SecondOrderVariant):
    """r taken as h_k / h_{k-1}."""
    def combine(self, x0, prev_x0, r):
        r = 1.0 / r
        return (1.0 + 1.0 / (2.0 * r)) * x0 - (1.0 / (2.0 * r)) * prev_x0


class _FlippedSign(_SecondOrderVariant):
    """D = (1 - 1/(2r)) x0_k + (1/(2r)) x0_{k-1}."""
    def combine(self, x0, prev_x0, r):
        return (1.0 - 1.0 / (2.0 * r)) * x0 + (1.0 / (2.0 * r)) * prev_x0


def _midpoint_error(cls, S=20):
    """max over second-order steps of |D - x0(lambda_k + h_k/2)| for an affine
    data prediction x0(lambda) = a + b lambda; D is read off the update
    x_{k+1} = (sigma_{k+1}/sigma_k) x_k + alpha_{k+1} (1 - e^{-h_k}) D."""
    smp = cls("dpmpp2m", S, 4)
    g = np.random.default_rng(21)
    a, b = g.normal(size=(1, 4, 2, 2)), g.normal(size=(1, 4, 2, 2))
    x = g.normal(size=(1, 4, 2, 2))
    worst = 0.0
    for k in range(S - 1):
        al, sg, lam = _alpha_sigma_lambda(smp, k)
        al2, sg2, lam2 = _alpha_sigma_lambda(smp, k + 1)
        h = lam2 - lam
        x_next = smp.step(k, x, _eps_for(smp, k, x, a + b * lam))
        D = (x_next - (sg2 / sg) * x) / (al2 * (1.0 - math.exp(-h)))
        want = a + b * (lam + (h / 2.0 if k > 0 else 0.0))
        worst = max(worst, float(np.abs(D - want).max() / np.abs(want).max()))
        x = x_next
    return worst


def test_dpmpp2m_combined_estimate_is_the_midpoint_for_affine_predictions():
    assert _midpoint_error(osm.Sampler) <= 1e-11


def _ode_error(kind, S, cls=osm.Sampler):
    """Error after S/2 steps (model time 499 for every even S) against the
    closed-form solution of the probability-flow ODE in data-prediction form,
    x(l) = (sigma/sigma_s) x_s + sigma * integral_{l_s}^{l} e^u x0(u) du, for
    x0(u) = sin(u) (elementwise constant): the integral of e^u sin u is
    e^u (sin u - cos u) / 2."""
    smp = cls(kind, S, 1)
    x = np.full((1, 1, 1, 1), 0.3)
    _, sg0, l0 = _alpha_sigma_lambda(smp, 0)
    for k in range(S // 2):
        lam = _alpha_sigma_lambda(smp, k)[2]
        x = smp.step(k, x, _eps_for(smp, k, x, np.sin(lam)))
    assert smp.tau[S // 2] == 499
    _, sg, l1 = _alpha_sigma_lambda(smp, S // 2)
    prim = lambda u: math.exp(u) * (math.sin(u) - math.cos(u)) / 2.0
    exact = (sg / sg0) * 0.3 + sg * (prim(l1) - prim(l0))
    return abs(float(x.ravel()[0]) - exact)


def test_global_order_dpmpp2m_second_ddim_first():
    Ss = [20, 40, 80, 160]
    ddim = [_ode_error("ddim", S) for S in Ss]
    dpm = [_ode_error("dpmpp2m", S) for S in Ss]
    rd = [ddim[i] / ddim[i + 1] for i in range(3)]
    rp = [dpm[i] / dpm[i + 1] for i in range(3)]
    print("ddim error ratios", rd, "dpm++(2m)", rp)
    assert all(1.7 < r < 2.3 for r in rd[1:]), rd
    assert all(3.4 < r < 4.6 for r in rp[1:]), rp
    assert dpm[-1] < ddim[-1] / 10


def _golden_dpm():
    rows = {}
    with open(os.path.join(HERE, "golden", "dpmpp2m_worked.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                key, *vals = line.split()
                rows[key] = [float(v) for v in vals]
    return rows


def _golden_run(cls):
    gd = _golden_dpm()
    smp = cls("dpmpp2m", 4, 1)
    smp.ab = np.array(gd["alpha_bar"])          # the worked example's own schedule
    smp.tau = np.arange(4)
    x = np.full((1, 1, 1, 1), gd["x_start"][0])
    xs = []
    for k, x0 in enumerate(gd["x0_pred"]):
        x = smp.step(k, x, _eps_for(smp, k, x, np.full_like(x, x0)))
        xs.append(float(x.ravel()[0]))
    return xs, gd["x_after"]


def test_dpmpp2m_two_step_worked_example():
    got, exp = _golden_run(osm.Sampler)
    np.testing.assert_allclose(got, exp, rtol=1e-13, atol=1e-14)


def test_planted_sampler_mistakes_fail_the_pins():
    assert _midpoint_error(_InvertedR) > 1e-3
    assert _midpoint_error(_FlippedSign) > 1e-3
    for cls in (_InvertedR, _FlippedSign):
        got, exp = _golden_run(cls)
        assert abs(got[2] - exp[2]) > 1e-3, cls.__name__
