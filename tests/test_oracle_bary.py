"""Pins for the oracle's barycentric weights, mask, ring/plan and forecast.

Each check ties the oracle to something other than itself: values the paper
prints (its FLOPs columns), closed forms worked by hand, exact rational
Lagrange interpolation, polynomial reproduction, and invariants.
"""
import collections
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import bary

HERE = os.path.dirname(os.path.abspath(__file__))


def _golden(name):
    rows = []
    with open(os.path.join(HERE, "golden", name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line)
    return rows


def _params(C=math.inf, eta=0.0, delta=1.0, lam=0.0, nodes="trapezoid", blend="recent"):
    return bary.Params(nodes=nodes, C=C, eta=eta, delta=delta, lam=lam, blend=blend)


@pytest.mark.parametrize("row", _golden("bary_worked.txt"))
def test_worked_values(row):
    f = [x.strip() for x in row.split("|")]
    s = [float(v) for v in f[0].split(",")]
    t, C, eta, delta, lam = (float(v) for v in f[1:6])
    w = bary.bary_weights(s, t, _params(C=C, eta=eta, delta=delta, lam=lam, blend=f[6]))
    exp = np.array([float(v) for v in f[7].split(",")])
    np.testing.assert_allclose(w, exp, rtol=1e-13, atol=1e-14)


def test_k2_is_linear_extrapolation():
    g = np.random.default_rng(1)
    for _ in range(200):
        s2, s1 = np.sort(g.uniform(-5, 5, 2))
        t = s1 + g.uniform(0.6, 3.0)      # beyond the newest node
        w = bary.bary_weights([s1, s2], t, _params(C=math.inf))
        exp = [(t - s2) / (s1 - s2), (s1 - t) / (s1 - s2)]
        np.testing.assert_allclose(w, exp, rtol=1e-12, atol=1e-12)


def test_k3_equispaced_reproduces_quadratics_at_delta1():
    g = np.random.default_rng(2)
    for _ in range(100):
        h = g.uniform(0.5, 3.0)
        s0 = g.uniform(-3, 3)
        s = [s0 + 2 * h, s0 + h, s0]
        t = s[0] + g.uniform(0.2, 2.0) * h
        a, b, c = g.normal(size=3)
        f = lambda x: a + b * x + c * x * x
        w = bary.bary_weights(s, t, _params(C=math.inf))
        assert abs(np.dot(w, [f(x) for x in s]) - f(t)) < 1e-10 * (1 + abs(f(t)))


def test_k3_paper_delta_is_not_exact_but_sums_to_one():
    s, t = [8.0, 4.0, 0.0], 9.0
    w = bary.bary_weights(s, t)                 # paper defaults: C=10, delta_3 = 0.95
    assert abs(w.sum() - 1.0) < 1e-14
    exact = np.array([1.40625, -0.5625, 0.15625])
    assert np.max(np.abs(w - exact)) > 1e-3


def test_k4_trapezoid_is_floater_hormann_d1():
    """Sec. 3.2 identifies the trapezoid weights on equispaced nodes with the
    Floater-Hormann interpolant of degree d <= 1: it reproduces linear
    functions (and, being of degree 1, not quadratics)."""
    s = [3.0, 2.0, 1.0, 0.0]
    for t in (3.5, 4.0, 5.25):
        w = bary.bary_weights(s, t, _params(C=math.inf))
        for a, b in ((0.3, -1.2), (2.0, 0.5)):
            assert abs(np.dot(w, [a + b * x for x in s]) - (a + b * t)) < 1e-12
        assert abs(np.dot(w, [x * x for x in s]) - t * t) > 1e-3


def _lagrange_fraction(s, t):
    s = [Fraction(v) for v in s]
    t = Fraction(t)
    out = []
    for j in range(len(s)):
        num, den = Fraction(1), Fraction(1)
        for m in range(len(s)):
            if m != j:
                num *= t - s[m]
                den *= s[j] - s[m]
        out.append(num / den)
    return out


def test_lagrange_mode_matches_rational_brute_force():
    g = np.random.default_rng(3)
    for K in range(1, 7):
        for _ in range(30):
            s = list(g.choice(np.arange(-20, 21), size=K, replace=False).astype(float))
            t = float(g.integers(-25, 26)) + 0.5
            w = bary.bary_weights(s, t, _params(nodes="lagrange"))
            exp = np.array([float(v) for v in _lagrange_fraction(s, t)])
            np.testing.assert_allclose(w, exp, rtol=1e-10, atol=1e-10 * np.abs(exp).max())


def test_lagrange_mode_reproduces_degree_below_k_and_node_values():
    g = np.random.default_rng(4)
    for K in range(1, 8):
        s = sorted(g.uniform(0, 10, K), reverse=True)
        coef = g.normal(size=K)
        f = lambda x: sum(c * x ** i for i, c in enumerate(coef))
        t = s[0] + 1.3
        w = bary.bary_weights(s, t, _params(nodes="lagrange"))
        assert abs(np.dot(w, [f(x) for x in s]) - f(t)) < 1e-8 * (1 + abs(f(t)))
        for j in range(K):
            wj = bary.bary_weights(s, s[j], _params(nodes="lagrange"))
            assert list(wj) == [1.0 if i == j else 0.0 for i in range(K)]


def test_weights_sum_to_one_and_blend():
    g = np.random.default_rng(5)
    for K in range(1, 9):
        for _ in range(20):
            s = list(np.sort(g.uniform(0, 1, K)))          # increasing: newest first
            t = s[0] - g.uniform(0.01, 0.3)
            try:
                w = bary.bary_weights(s, t)
            except bary.Degenerate:
                continue
            assert abs(w.sum() - 1.0) < 1e-12 * max(1.0, np.abs(w).sum())
            w1 = bary.bary_weights(s, t, bary.Params(lam=1.0))
            assert list(w1) == [1.0] + [0.0] * (K - 1)


def test_literal_blend_option():
    w = bary.bary_weights([4.0, 0.0], 5.0, _params(C=10, blend="literal", lam=0.0))
    assert list(w) == [1.25, 0.0]
    w = bary.bary_weights([4.0, 0.0], 5.0, _params(C=10, blend="literal", lam=1.0))
    assert list(w) == [0.0, -0.25]


def test_affine_invariance_without_clip():
    g = np.random.default_rng(6)
    for K in range(2, 6):
        s = list(np.arange(K, 0, -1) * 1.0)
        t = K + 0.7
        for delta in (1.0, 0.95, 0.7):
            w = bary.bary_weights(s, t, _params(delta=delta))
            a, b = g.uniform(0.1, 50), g.uniform(-100, 100)
            w2 = bary.bary_weights([a * x + b for x in s], a * t + b, _params(delta=delta))
            np.testing.assert_allclose(w, w2, rtol=1e-12, atol=1e-13)


def test_node_order_reversal_symmetry():
    """Trapezoid coefficients are symmetric, so reversing the node order only
    flips every sign of u, which the normalisation removes."""
    s, t = [3.0, 2.0, 1.0, 0.0], 3.6
    w = bary.bary_weights(s, t)
    wr = bary.bary_weights(s[::-1], t)
    np.testing.assert_allclose(w, wr[::-1], rtol=1e-14)


def test_query_on_node_is_clipped_in_trapezoid_mode():
    w = bary.bary_weights([1.0, 0.0], 1.0, _params(C=10))
    # u1 = -0.5/0 -> -inf -> -10; u2 = 0.5/1
    a1 = 10 / (10 - 0.5)
    np.testing.assert_allclose(w, [a1, 1 - a1], rtol=1e-14)


def test_degenerate_when_clipped_terms_cancel():
    with pytest.raises(bary.Degenerate):
        bary.bary_weights([0.5, 0.52], 0.49)          # both |u| > C, opposite signs


@pytest.mark.parametrize("bad", [([], 1.0), ([1.0] * 9, 2.0), ([1.0, 1.0], 2.0),
                                 ([0.0, 2.0, 1.0], 3.0), ([math.nan], 1.0)])
def test_invalid_nodes(bad):
    with pytest.raises(ValueError):
        bary.bary_weights(*bad)


def test_delta_table_is_the_papers():
    assert (bary.delta_for(2), bary.delta_for(3), bary.delta_for(4)) == (1.0, 0.95, 0.7)
    assert bary.CLIP_C == 10.0 and bary.ETA == 1e-12


# ---------------------------------------------------------------------------
# mask, ring, plan, forecast
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("row", _golden("paper_flops.txt"))
def test_mask_full_step_count_matches_paper_flops(row):
    model, N, flops, vanilla, _src = row.split()
    implied = round(50 * float(flops) / float(vanilla))
    assert int(bary.make_mask(50, int(N)).sum()) == implied


def test_mask_shapes():
    assert list(np.nonzero(bary.make_mask(10, 3))[0]) == [0, 3, 6, 9]
    assert list(np.nonzero(bary.make_mask(20, 4))[0]) == [0, 4, 8, 12, 16, 19]
    assert bary.make_mask(50, 5).sum() == 11
    assert bary.make_mask(7, 1).sum() == 7


def test_ring_matches_a_deque_model():
    g = np.random.default_rng(7)
    for K in range(1, 9):
        for _ in range(20):
            S = int(g.integers(1, 40))
            mask = (g.uniform(size=S) < 0.4).astype(np.uint8)
            mask[0] = 1
            steps = bary.plan(mask, K)
            dq = collections.deque(maxlen=K)
            slot_of = {}
            ring = bary.Ring(K)
            for k in range(S):
                if mask[k]:
                    dq.appendleft(k)
                    slot_of[k] = ring.push(None, k)
                    assert steps[k].is_full and steps[k].head == slot_of[k]
                    assert steps[k].count == len(dq)
                else:
                    st = steps[k]
                    assert not st.is_full and st.count == len(dq)
                    assert [slot_of[n] for n in dq] == st.slots
                    exp = bary.bary_weights([float(n) for n in dq], float(k))
                    assert list(exp) == st.w


def test_plan_rejects_mask_without_first_full_step():
    with pytest.raises(ValueError):
        bary.plan([0, 1, 1], 2)


def test_forecast_is_exact_weighted_sum():
    g = np.random.default_rng(8)
    for K in range(1, 6):
        feats = [g.integers(-1000, 1000, size=7) / 64.0 for _ in range(K)]
        w = [g.integers(-64, 64) / 32.0 for _ in range(K)]
        got = bary.forecast(feats, w)
        for i in range(7):
            exact = sum(Fraction(w[j]) * Fraction(feats[j][i]) for j in range(K))
            assert got[i] == float(exact)
