"""Pins for the oracle's blockwise mode (Br = 0; Sec. 4.5, Tables 5 and 6).

* With every step full there is nothing to forecast: the run is the stepwise
  loop's, bit for bit.
* The module sites and their gates rebuild the stack's output: the embedding
  plus the gated module outputs, summed, is the full step's feature.
* With gates constant in time (zero modulation weights), the forecast is
  linear and the embedding affine with weights summing to one, so a skipped
  step's feature must be the stepwise forecast of the full steps' features
  plus the current embedding minus the forecast of the nodes' embeddings.
  With time-varying gates that identity must fail: the current gates are used.
"""

import numpy as np
import pytest

import synth
from oracle import bary, model as om, sampler as osm


def _pixart_small():
    return synth.scaled(synth.CONFIGS["pixart"], depth=2, hidden=64, heads=2, head_dim=32, mlp=128,
                        latent=(4, 8, 8), batch=2, ctx_tokens=5, ctx_dim=16, steps=10, dtype="f32")


def _setup(kind, const_gates=False):
    cfg = synth.CONFIGS["tiny"] if kind == "dit" else _pixart_small()
    P = dict(synth.params(cfg))
    if const_gates:
        for l in range(cfg.depth):
            if kind == "dit":
                P[f"blocks.{l}.w_mod"] = np.zeros_like(P[f"blocks.{l}.w_mod"])
        if kind == "pixart":
            P["t6_w"] = np.zeros_like(P["t6_w"])
    M = om.Model(cfg, P)
    xT = synth.latents(cfg).astype(np.float64)
    text = synth.text(cfg) if kind == "pixart" else None
    return cfg, M, xT, text


@pytest.mark.parametrize("kind", ["dit", "pixart"])
def test_all_full_is_the_stepwise_loop(kind):
    cfg, M, xT, text = _setup(kind)
    mask = np.ones(cfg.steps, np.uint8)
    assert np.array_equal(osm.sample_blockwise(M, xT, mask, cfg.K, text=text),
                          osm.sample(M, xT, mask, cfg.K, text=text))


@pytest.mark.parametrize("kind", ["dit", "pixart"])
def test_sites_rebuild_the_stack(kind):
    cfg, M, xT, text = _setup(kind)
    tin = osm.model_time(cfg.sampler, cfg.steps)
    cond = M.condition(tin[3], xT.shape[0], None, text)
    ctx = M.context(text) if text is not None else None
    emb = M.embed(xT)
    h, sites, gates = emb, [], []
    for l in range(cfg.depth):
        mod = M.block_mod(l, cond)
        h = M.dit_block(l, h, mod, ctx, modules=sites)
        gates += M.module_gates(l, mod)
    assert len(sites) == len(gates) == cfg.depth * (3 if kind == "pixart" else 2)
    rebuilt = emb + sum(g[:, None, :] * m for g, m in zip(gates, sites))
    np.testing.assert_allclose(rebuilt, h, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(h, M.stack(emb, cond, ctx))


def _identity_gap(cfg, M, xT, text):
    mask = bary.make_mask(cfg.steps, cfg.interval)
    tr = {}
    osm.sample_blockwise(M, xT, mask, cfg.K, text=text, trace=tr)
    steps = bary.plan(mask, cfg.K)
    full = [k for k in range(cfg.steps) if mask[k]]
    gaps = []
    for k in range(cfg.steps):
        if mask[k]:
            continue
        st = steps[k]
        held = [f for f in full if f < k][-st.count:][::-1]        # the nodes: newest first
        fc_feat = bary.forecast([tr["feat"][f] for f in held], st.w)
        fc_emb = bary.forecast([tr["emb"][f] for f in held], st.w)
        pred = fc_feat + tr["emb"][k] - fc_emb
        gaps.append(np.linalg.norm(tr["feat"][k] - pred) / np.linalg.norm(tr["feat"][k]))
    return max(gaps)


@pytest.mark.parametrize("kind", ["dit", "pixart"])
def test_constant_gates_make_it_a_shifted_stepwise_forecast(kind):
    cfg, M, xT, text = _setup(kind, const_gates=True)
    assert _identity_gap(cfg, M, xT, text) < 1e-12


@pytest.mark.parametrize("kind", ["dit", "pixart"])
def test_time_varying_gates_are_applied(kind):
    cfg, M, xT, text = _setup(kind)
    assert _identity_gap(cfg, M, xT, text) > 1e-6


def test_rejects_mmdit():
    cfg = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=64, heads=2, head_dim=32,
                       mlp=128, latent=(16, 2, 4, 6), txt_tokens=3)
    with pytest.raises(ValueError):
        osm.sample_blockwise(om.Model(cfg, synth.params(cfg)), synth.latents(cfg).astype(np.float64),
                             bary.make_mask(6, 5), 3, text=synth.text(cfg))
