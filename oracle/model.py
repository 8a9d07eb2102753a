"""Oracle: the DiT-family denoiser whose block stack BaryCache skips.

TEST INFRASTRUCTURE ONLY (tests, smoke check and the benchmark's CPU baseline
import it).  Plain numpy, fp64 by default, no blocking or fusion.  Shares no
code with the HIP library.

The paper fixes only the structure of the stack (Sec. 3.1, Eqs. 4-5): a token
embedding of the noisy input with conditioning and timestep embeddings fused
in, L layers of residual modules, and the stepwise feature x'_t, which is the
output of the whole layer stack and the thing BaryCache caches.  It evaluates
DiT-XL/2, PixArt-Sigma and HunyuanVideo (Sec. 4.1) but prints none of their
internals, so the block internals below are the standard published
architectures written out as math, with these readings:
  * Eq. 4's residual is the running residual stream: each module adds its
    output to the stream it read;
  * DiT block (adaLN-Zero form, random non-zero parameters): six modulation
    vectors (shift1, scale1, gate1, shift2, scale2, gate2) from SiLU(c);
    LayerNorm without affine, eps 1e-6; GELU with the tanh approximation;
  * PixArt block: the six vectors are t6 + a per-block table; a cross-attention
    to the projected caption follows self-attention, without norm or gate;
  * dual-stream block: image and text streams each with their own modulation,
    projections and MLP, attention joint over the concatenated tokens; single-
    stream block: one fused projection to [qkv | mlp], one fused output
    projection of [attention | GELU(mlp)], one gate; queries and keys take a
    per-head RMSNorm and a 3D rotary embedding of the image tokens (Model.qk).
    The token refiner and guidance embedding are left out;
  * the cached feature is the image-token part of the last block's output; the
    final layer runs on every step, full or forecast.
"""
from __future__ import annotations

import math
from typing import Dict, Optional, Tuple

import numpy as np

LN_EPS = 1e-6


def silu(x):
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x):
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def layer_norm(x, eps=LN_EPS):
    """Normalise the last axis: (x - mean) / sqrt(biased variance + eps)."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def rms_norm(x, w, eps=LN_EPS):
    """RMSNorm over the last axis with a learned scale: x / sqrt(mean(x^2) + eps) * w."""
    return x / np.sqrt((x * x).mean(-1, keepdims=True) + eps) * w


def rope_axes(head_dim):
    """Head dimensions given to the (frame, row, column) axes of the 3D rotary
    embedding: head_dim/8 to the frame index and the rest split evenly between
    row and column (128 -> 16, 56, 56, the split of the video model's 3D RoPE)."""
    dt = head_dim // 8
    dh = (head_dim - dt) // 2
    axes = (dt, dh, head_dim - dt - dh)
    if any(d % 2 for d in axes):
        raise ValueError("the 3D rotary embedding needs head_dim % 32 == 0")
    return axes


def rope_angles(grid, head_dim, theta):
    """Rotation angle of every (token, pair) [T, head_dim/2] for a (F, H, W)
    token grid in (frame, row, column) order.  Pair i holds dimensions 2i and
    2i + 1; in an axis of d dimensions its j-th pair turns by
    pos * theta^(-2j / d), pos being the token's index along that axis."""
    F, H, W = grid
    f, h, w = np.meshgrid(np.arange(F), np.arange(H), np.arange(W), indexing="ij")
    pos = [f.reshape(-1), h.reshape(-1), w.reshape(-1)]
    cols = []
    for p_a, d in zip(pos, rope_axes(head_dim)):
        freq = theta ** (-np.arange(0, d, 2, dtype=np.float64) / d)
        cols.append(p_a[:, None].astype(np.float64) * freq[None, :])
    return np.concatenate(cols, axis=1)


def apply_rope(x, ang):
    """Rotate each pair (x[..., 2i], x[..., 2i+1]) of x [..., T, head_dim] by
    ang [T, head_dim/2]."""
    c, s = np.cos(ang), np.sin(ang)
    x0, x1 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x0 * c - x1 * s
    out[..., 1::2] = x0 * s + x1 * c
    return out


def modulate(h, shift, scale):
    """h * (1 + scale) + shift, with per-sample [B, D] vectors broadcast over tokens."""
    return h * (1.0 + scale[:, None, :]) + shift[:, None, :]


def linear(x, w, b=None):
    y = x @ w.T
    if b is not None:
        y = y + b
    return y


def attention(q, k, v):
    """softmax(q k^T / sqrt(d)) v for [B, H, Tq, d] queries and [B, H, Tk, d] keys/values."""
    d = q.shape[-1]
    out = np.empty(q.shape[:-1] + (v.shape[-1],), dtype=q.dtype)
    for b in range(q.shape[0]):
        for h in range(q.shape[1]):
            s = (q[b, h] @ k[b, h].T) / math.sqrt(d)
            s = s - s.max(axis=-1, keepdims=True)
            e = np.exp(s)
            out[b, h] = (e / e.sum(axis=-1, keepdims=True)) @ v[b, h]
    return out


def split_heads(x, heads):
    B, T, D = x.shape
    return x.reshape(B, T, heads, D // heads).transpose(0, 2, 1, 3)


def merge_heads(x):
    B, H, T, d = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B, T, H * d)


def timestep_embedding(tau, dim=256, dtype=np.float64):
    """[cos(tau f_i), sin(tau f_i)] with f_i = 10000^(-i/(dim/2)), i < dim/2.

    `tau` is a scalar or a [B] vector of model time inputs."""
    half = dim // 2
    f = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    a = np.atleast_1d(np.asarray(tau, dtype=np.float64))[:, None] * f[None, :]
    return np.concatenate([np.cos(a), np.sin(a)], axis=-1).astype(dtype)


def patchify(lat, p):
    """[B, C, (F,) H, W] -> [B, T, p*p*C], tokens row-major over (F,) H/p, W/p,
    features ordered (p_h, p_w, c)."""
    if lat.ndim == 4:
        B, C, H, W = lat.shape
        x = lat.reshape(B, C, H // p, p, W // p, p)
        x = x.transpose(0, 2, 4, 3, 5, 1)          # B, h, w, ph, pw, C
        return x.reshape(B, (H // p) * (W // p), p * p * C)
    B, C, F, H, W = lat.shape
    x = lat.reshape(B, C, F, H // p, p, W // p, p)
    x = x.transpose(0, 2, 3, 5, 4, 6, 1)           # B, f, h, w, ph, pw, C
    return x.reshape(B, F * (H // p) * (W // p), p * p * C)


def unpatchify(tok, p, latent_shape, C_out):
    """Exact inverse of `patchify` for C_out channels."""
    if len(latent_shape) == 3:
        _, H, W = latent_shape
        B = tok.shape[0]
        x = tok.reshape(B, H // p, W // p, p, p, C_out).transpose(0, 5, 1, 3, 2, 4)
        return x.reshape(B, C_out, H, W)
    _, F, H, W = latent_shape
    B = tok.shape[0]
    x = tok.reshape(B, F, H // p, W // p, p, p, C_out).transpose(0, 6, 1, 2, 4, 3, 5)
    return x.reshape(B, C_out, F, H, W)


class Model:
    """The denoiser of one synthetic workload (a `synth.ModelConfig`) with
    explicit parameters (name -> array).  Computes in `dtype` (fp64 default)."""

    def __init__(self, cfg, params: Dict[str, np.ndarray], dtype=np.float64):
        self.cfg = cfg
        self.dt = dtype
        self.P = {k: np.asarray(v, dtype=dtype) for k, v in params.items()}

    # -- conditioning --------------------------------------------------------
    def t_embed(self, tau, B):
        P = self.P
        e = timestep_embedding(np.full(B, tau, dtype=np.float64), self.cfg.freq_dim, self.dt)
        return linear(silu(linear(e, P["t_w1"], P["t_b1"])), P["t_w2"], P["t_b2"])

    def condition(self, tau, B, labels=None, text=None):
        """Per-step conditioning: returns a dict with 'c' (and 't6' for pixart)."""
        cfg, P = self.cfg, self.P
        t = self.t_embed(tau, B)
        out = {"t": t}
        if cfg.kind == "dit":
            c = t
            if cfg.n_classes:
                c = t + P["y_table"][np.asarray(labels)]
            out["c"] = c
        elif cfg.kind == "pixart":
            out["c"] = t
            out["t6"] = linear(silu(t), P["t6_w"], P["t6_b"])
        else:
            pooled = np.asarray(text, dtype=self.dt).mean(axis=1)
            out["c"] = t + linear(pooled, P["txt_w"], P["txt_b"])
        return out

    def context(self, text):
        """Per-run text context.  pixart: caption projection and every block's
        cross-attention keys/values, which do not depend on the step."""
        cfg, P = self.cfg, self.P
        text = np.asarray(text, dtype=self.dt)
        if cfg.kind != "pixart":
            return {"txt": text}
        ctx = linear(gelu_tanh(linear(text, P["cap_w1"], P["cap_b1"])), P["cap_w2"], P["cap_b2"])
        kv = []
        D = cfg.hidden
        for l in range(cfg.depth):
            y = linear(ctx, P[f"blocks.{l}.wx_kv"], P[f"blocks.{l}.bx_kv"])
            kv.append((split_heads(y[..., :D], cfg.heads), split_heads(y[..., D:], cfg.heads)))
        return {"ctx": ctx, "kv": kv}

    # -- embedding and final layer ---------------------------------------------
    def embed(self, lat):
        P = self.P
        tok = patchify(np.asarray(lat, dtype=self.dt), self.cfg.p)
        return linear(tok, P["patch_w"], P["patch_b"]) + P["pos"][None]

    def final(self, feat, cond):
        """Final layer: adaLN (shift, scale), LayerNorm, linear to p*p*C_out,
        unpatchify.  Runs on the cached or forecast feature alike."""
        cfg, P = self.cfg, self.P
        D = cfg.hidden
        if cfg.kind == "pixart":
            shift = P["final_table"][0][None] + cond["t"]
            scale = P["final_table"][1][None] + cond["t"]
        else:
            m = linear(silu(cond["c"]), P["final_w_mod"], P["final_b_mod"])
            shift, scale = m[:, :D], m[:, D:]
        h = modulate(layer_norm(np.asarray(feat, dtype=self.dt)), shift, scale)
        y = linear(h, P["final_w"], P["final_b"])
        return unpatchify(y, cfg.p, cfg.latent, cfg.out_ch)

    # -- query/key processing of the video model's blocks -------------------------
    def token_grid(self):
        cfg = self.cfg
        if len(cfg.latent) == 3:
            return 1, cfg.latent[1] // cfg.p, cfg.latent[2] // cfg.p
        return cfg.latent[1], cfg.latent[2] // cfg.p, cfg.latent[3] // cfg.p

    def qk(self, q, k, pre, n_img):
        """RMSNorm (per head, learned scales pre+q_norm / pre+k_norm) and the 3D
        rotary embedding of the first n_img tokens, on q, k [B, H, T, hd]."""
        cfg, P = self.cfg, self.P
        if cfg.qk_norm:
            q = rms_norm(q, P[pre + "q_norm"])
            k = rms_norm(k, P[pre + "k_norm"])
        if cfg.rope_theta and n_img:
            ang = rope_angles(self.token_grid(), cfg.head_dim, cfg.rope_theta)
            q, k = q.copy(), k.copy()
            q[:, :, :n_img] = apply_rope(q[:, :, :n_img], ang)
            k[:, :, :n_img] = apply_rope(k[:, :, :n_img], ang)
        return q, k

    # -- blocks ----------------------------------------------------------------
    def block_mod(self, l, cond):
        """The six [B, D] modulation vectors of DiT/PixArt block l."""
        cfg, P = self.cfg, self.P
        D = cfg.hidden
        if cfg.kind == "pixart":
            m = cond["t6"] + P[f"blocks.{l}.table"].reshape(1, 6 * D)
        else:
            m = linear(silu(cond["c"]), P[f"blocks.{l}.w_mod"], P[f"blocks.{l}.b_mod"])
        return [m[:, i * D:(i + 1) * D] for i in range(6)]

    def dit_block(self, l, x, mod, ctx=None, modules=None, rows=None):
        """One DiT (or PixArt) block on the residual stream x [B, T, D].
        `modules`, if a list, receives the block's module outputs before their
        gates (attention, PixArt's cross-attention, MLP): the sites that
        blockwise caching keeps (Sec. 3.1, Eq. 4: the increments M_q).
        `rows`, if given, is a list of token indices: keys and values still
        come from every token, but only those tokens' outputs are computed and
        returned ([B, len(rows), D]); every other step is per token."""
        cfg, P = self.cfg, self.P
        pre = f"blocks.{l}."
        s1, sc1, g1, s2, sc2, g2 = mod
        D, H = cfg.hidden, cfg.heads
        h = modulate(layer_norm(x), s1, sc1)
        qkv = linear(h, P[pre + "w_qkv"], P[pre + "b_qkv"])
        q, k, v = (split_heads(qkv[..., i * D:(i + 1) * D], H) for i in range(3))
        if rows is not None:
            x, q = x[:, rows], q[:, :, rows]
        a = merge_heads(attention(q, k, v))
        o = linear(a, P[pre + "w_o"], P[pre + "b_o"])
        x = x + g1[:, None, :] * o
        outs = [o]
        if cfg.kind == "pixart":
            kx, vx = ctx["kv"][l]
            qx = split_heads(linear(x, P[pre + "wx_q"], P[pre + "bx_q"]), H)
            o = linear(merge_heads(attention(qx, kx, vx)), P[pre + "wx_o"], P[pre + "bx_o"])
            x = x + o
            outs.append(o)
        h = modulate(layer_norm(x), s2, sc2)
        m = gelu_tanh(linear(h, P[pre + "w_fc1"], P[pre + "b_fc1"]))
        o = linear(m, P[pre + "w_fc2"], P[pre + "b_fc2"])
        outs.append(o)
        if modules is not None:
            modules.extend(outs)
        return x + g2[:, None, :] * o

    def module_gates(self, l, mod):
        """The gates of block l's module sites, in the order dit_block records
        them (the cross-attention of PixArt has none: a gate of one)."""
        g1, g2 = mod[2], mod[5]
        if self.cfg.kind == "pixart":
            return [g1, np.ones_like(g1), g2]
        return [g1, g2]

    def dual_block(self, l, xi, xt, cond, rows=None):
        """Dual-stream block on image tokens xi [B, Ti, D] and text tokens
        xt [B, Tt, D]; returns both streams.  `rows` = (image rows, text rows):
        only those tokens' outputs are computed (keys and values from all)."""
        cfg, P = self.cfg, self.P
        D, H = cfg.hidden, cfg.heads
        Ti = xi.shape[1]
        mods, qs, ks, vs = {}, [], [], []
        for s, x in (("img", xi), ("txt", xt)):
            pre = f"dual.{l}.{s}."
            m = linear(silu(cond["c"]), P[pre + "w_mod"], P[pre + "b_mod"])
            mods[s] = [m[:, i * D:(i + 1) * D] for i in range(6)]
            h = modulate(layer_norm(x), mods[s][0], mods[s][1])
            qkv = linear(h, P[pre + "w_qkv"], P[pre + "b_qkv"])
            q, k, v = (split_heads(qkv[..., i * D:(i + 1) * D], H) for i in range(3))
            q, k = self.qk(q, k, pre, Ti if s == "img" else 0)
            qs.append(q)
            ks.append(k)
            vs.append(v)
        q, k, v = (np.concatenate(z, axis=2) for z in (qs, ks, vs))
        if rows is not None:
            ri, rt = list(rows[0]), list(rows[1])
            q = q[:, :, ri + [Ti + r for r in rt]]
            xi, xt, Ti = xi[:, ri], xt[:, rt], len(ri)
        a = merge_heads(attention(q, k, v))
        outs = []
        for s, x, a_s in (("img", xi, a[:, :Ti]), ("txt", xt, a[:, Ti:])):
            pre = f"dual.{l}.{s}."
            s1, sc1, g1, s2, sc2, g2 = mods[s]
            x = x + g1[:, None, :] * linear(a_s, P[pre + "w_o"], P[pre + "b_o"])
            h = modulate(layer_norm(x), s2, sc2)
            mm = gelu_tanh(linear(h, P[pre + "w_fc1"], P[pre + "b_fc1"]))
            outs.append(x + g2[:, None, :] * linear(mm, P[pre + "w_fc2"], P[pre + "b_fc2"]))
        return outs[0], outs[1]

    def single_block(self, l, x, cond, n_img=0, rows=None):
        """Single-stream block on x [B, T_img + T_txt, D] (the first n_img
        tokens are image tokens).  `rows`: token indices whose outputs alone
        are computed (keys and values from all tokens)."""
        cfg, P = self.cfg, self.P
        D, H = cfg.hidden, cfg.heads
        pre = f"single.{l}."
        m = linear(silu(cond["c"]), P[pre + "w_mod"], P[pre + "b_mod"])
        s, sc, g = m[:, :D], m[:, D:2 * D], m[:, 2 * D:]
        h = modulate(layer_norm(x), s, sc)
        y = linear(h, P[pre + "w_1"], P[pre + "b_1"])
        q, k, v = (split_heads(y[..., i * D:(i + 1) * D], H) for i in range(3))
        q, k = self.qk(q, k, pre, n_img)
        if rows is not None:
            x, y, q = x[:, rows], y[:, rows], q[:, :, rows]
        a = merge_heads(attention(q, k, v))
        z = np.concatenate([a, gelu_tanh(y[..., 3 * D:])], axis=-1)
        return x + g[:, None, :] * linear(z, P[pre + "w_2"], P[pre + "b_2"])

    def probe(self, x, cond):
        """The feature an adaptive schedule watches: the first block's modulated
        attention input LN(x)(1 + scale1) + shift1 on the embedded latent x
        (image stream of the first dual block for MMDiT).  It costs the
        embedding, one modulation and one LayerNorm, not the stack."""
        cfg, P = self.cfg, self.P
        D = cfg.hidden
        if cfg.kind in ("dit", "pixart"):
            shift, scale = self.block_mod(0, cond)[:2]
        else:
            m = linear(silu(cond["c"]), P["dual.0.img.w_mod"], P["dual.0.img.b_mod"])
            shift, scale = m[:, :D], m[:, D:2 * D]
        return modulate(layer_norm(x), shift, scale)

    def stack(self, x, cond, ctx):
        """Eq. 5: the stepwise feature, i.e. the image-token output of the whole
        layer stack."""
        cfg = self.cfg
        if cfg.kind in ("dit", "pixart"):
            for l in range(cfg.depth):
                x = self.dit_block(l, x, self.block_mod(l, cond), ctx)
            return x
        xt = ctx["txt"]
        for l in range(cfg.depth):
            x, xt = self.dual_block(l, x, xt, cond)
        Ti = x.shape[1]
        z = np.concatenate([x, xt], axis=1)
        for l in range(cfg.depth_single):
            z = self.single_block(l, z, cond, Ti)
        return z[:, :Ti]
