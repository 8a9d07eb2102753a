"""Pins for the oracle's adaptive schedule (Sec. 4.5, Table 5): the decision
rule on hand-worked sequences, the probe's modulation chunk order, the relative
L1 change on a worked pair, the two limits of the threshold (every step full;
only the first and last), and that an adaptive run is the fixed-mask loop of
Sec. 3.3 under the mask it realised."""
import math
import os

import numpy as np
import pytest

import synth
from oracle import bary, model as om, sampler as osm

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "adaptive_rule.txt")


def _golden_cases():
    cases, cur = [], {}
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if not line:
            continue
        key, *vals = line.split()
        if key == "ell":
            cur = {"ell": float(vals[0])}
        elif key == "changes":
            cur["changes"] = [float(v) for v in vals]
        elif key == "mask":
            cur["mask"] = [int(v) for v in vals]
            cases.append(cur)
    return cases


@pytest.mark.parametrize("case", _golden_cases(), ids=lambda c: f"ell={c['ell']}")
def test_rule_hand_worked(case):
    assert osm.adaptive_mask(case["changes"], case["ell"]) == case["mask"]


def test_rule_rejects_bad_threshold():
    for ell in (-0.1, float("nan")):
        with pytest.raises(ValueError):
            osm.AdaptiveRule(ell, 5)


def test_rule_fewer_full_steps_for_larger_threshold():
    rng = np.random.default_rng(7)
    for _ in range(200):
        ch = rng.exponential(0.05, size=30)
        counts = [sum(osm.adaptive_mask(ch, ell)) for ell in (0.0, 0.02, 0.05, 0.1, 0.2, 0.5, math.inf)]
        assert counts[0] == 30 and counts[-1] == 2
        assert all(a >= b for a, b in zip(counts, counts[1:]))


def test_relative_l1_worked_pair():
    prev = np.array([1.0, -2.0, 3.0])
    cur = np.array([1.5, -2.0, 2.0])
    assert osm.relative_l1(cur, prev) == pytest.approx(1.5 / 6.0, rel=0, abs=1e-15)   # normalised by prev, not cur
    assert osm.relative_l1(prev, prev) == 0.0
    assert osm.relative_l1(np.zeros(3), np.zeros(3)) == 0.0
    assert osm.relative_l1(np.ones(3), np.zeros(3)) == math.inf


def _const_mod_params(cfg, prefix):
    """Zero modulation weights and a bias whose six D-chunks are the constants
    0.1, 0.2, ..., 0.6 (shift1, scale1, gate1, shift2, scale2, gate2)."""
    P = dict(synth.params(cfg))
    D = cfg.hidden
    P[prefix + "w_mod"] = np.zeros_like(P[prefix + "w_mod"])
    P[prefix + "b_mod"] = np.repeat(np.arange(1, 7) * 0.1, D)
    return P


@pytest.mark.parametrize("kind,prefix", [("tiny", "blocks.0."), ("hunyuan", "dual.0.img.")])
def test_probe_takes_the_first_shift_and_scale(kind, prefix):
    if kind == "tiny":
        cfg = synth.CONFIGS["tiny"]
    else:
        cfg = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=64, heads=2, head_dim=32,
                           mlp=128, latent=(16, 2, 4, 6), txt_tokens=3)
    P = _const_mod_params(cfg, prefix)
    m = om.Model(cfg, P)
    B = 2 if kind == "tiny" else 1
    x = np.random.default_rng(3).standard_normal((B, cfg.tokens, cfg.hidden))
    text = synth.text(cfg, batch=B) if cfg.kind != "dit" else None
    cond = m.condition(500.0, B, None, text)
    got = m.probe(x, cond)
    mu = x.mean(-1, keepdims=True)
    ln = (x - mu) / np.sqrt(((x - mu) ** 2).mean(-1, keepdims=True) + 1e-6)
    np.testing.assert_allclose(got, ln * 1.2 + 0.1, rtol=0, atol=1e-12)


def _tiny_run(ell):
    cfg = synth.CONFIGS["tiny"]
    m = om.Model(cfg, synth.params(cfg))
    xT = synth.latents(cfg).astype(np.float64)
    return cfg, m, xT, osm.sample_adaptive(m, xT, cfg.steps, ell, cfg.K)


def test_threshold_zero_is_the_all_full_loop():
    cfg, m, xT, (x, mask, ch) = _tiny_run(0.0)
    assert mask == [1] * cfg.steps
    assert np.array_equal(x, osm.sample(m, xT, mask, cfg.K))
    assert ch[0] == 0.0 and all(c > 0 for c in ch[1:])


def test_infinite_threshold_keeps_only_the_ends():
    cfg, m, xT, (x, mask, _) = _tiny_run(math.inf)
    assert mask == [1] + [0] * (cfg.steps - 2) + [1]
    assert np.array_equal(x, osm.sample(m, xT, mask, cfg.K))


@pytest.mark.parametrize("ell", [0.1, 0.3, 0.6])
def test_adaptive_run_is_the_fixed_loop_under_its_mask(ell):
    cfg, m, xT, (x, mask, ch) = _tiny_run(ell)
    assert 2 < sum(mask) < cfg.steps            # the threshold made a real choice
    assert np.array_equal(x, osm.sample(m, xT, mask, cfg.K))
    assert osm.adaptive_mask(ch, ell) == mask


def test_changes_are_the_probe_differences():
    cfg = synth.CONFIGS["tiny"]
    m = om.Model(cfg, synth.params(cfg))
    xT = synth.latents(cfg).astype(np.float64)
    tr = {}
    _, mask, ch = osm.sample_adaptive(m, xT, cfg.steps, 0.3, cfg.K, trace=tr)
    pr = tr["probe"]
    for k in range(1, cfg.steps):
        d = np.abs(pr[k] - pr[k - 1]).sum() / np.abs(pr[k - 1]).sum()
        assert ch[k] == pytest.approx(d, rel=1e-14)
    # the probe of step k is taken at the latent that step starts from
    tin = osm.model_time(cfg.sampler, cfg.steps)
    for k in (1, 5):
        cond = m.condition(tin[k], xT.shape[0])
        assert np.array_equal(pr[k], m.probe(m.embed(tr["x"][k - 1]), cond))
