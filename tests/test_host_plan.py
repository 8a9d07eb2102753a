"""The library's host logic (weights, mask, plan, schedule) against the oracle,
and the C ABI's exported symbols.  CPU only: none of these calls touch a GPU."""
import math
import os
import re
import subprocess

import numpy as np
import pytest

import synth
from oracle import bary, sampler as osm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _tol(w):
    return 1e-12 * max(1.0, float(np.abs(w).sum()))


def _lib_params(bc, p: bary.Params):
    return bc.params(nodes=p.nodes, clip_C=p.C, eta=p.eta, delta=p.delta, lam=p.lam, blend=p.blend)


def test_header_symbols_are_exported(bclib):
    hdr = open(os.path.join(ROOT, "include", "bc.h")).read()
    declared = set(re.findall(r"^\s*(?:int|void|size_t|const char\*)\s+(bc_\w+)\s*\(", hdr, re.M))
    assert len(declared) >= 20
    out = subprocess.run(["nm", "-D", "--defined-only", bclib.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (bc_\w+)$", out, re.M))
    assert declared <= exported, sorted(declared - exported)
    assert declared == set(bclib.exported_symbols())


def test_defaults_match_paper(bclib):
    p = bclib.default_params()
    assert (p.nodes, p.clip_C, p.eta, p.delta, p.lambda_, p.blend) == (0, 10.0, 1e-12, -1.0, 0.0, 0)


@pytest.mark.parametrize("mode", ["trapezoid", "lagrange"])
def test_weights_match_oracle_random(bclib, mode):
    g = np.random.default_rng(11)
    n = 0
    for K in range(1, 9):
        for _ in range(60):
            s = np.sort(g.uniform(0, 1, K))              # newest first: ascending, query below
            t = s[0] - g.uniform(0.001, 0.5)
            for C in (10.0, math.inf):
                for lam, blend in ((0.0, "recent"), (0.3, "recent"), (0.6, "literal")):
                    p = bary.Params(nodes=mode, C=C, lam=lam, blend=blend)
                    try:
                        exp = bary.bary_weights(s, t, p)
                    except bary.Degenerate:
                        with pytest.raises(bclib.BCError) as e:
                            bclib.bary_weights(s, t, _lib_params(bclib, p))
                        assert e.value.code == bclib.ERR_DEGENERATE
                        continue
                    got = bclib.bary_weights(s, t, _lib_params(bclib, p))
                    assert np.max(np.abs(got - exp)) <= _tol(exp)
                    n += 1
    assert n > 1000


def test_weights_worked_values(bclib):
    np.testing.assert_allclose(bclib.bary_weights([4.0, 0.0], 5.0), [1.25, -0.25], rtol=1e-10)  # eta-limited
    w = bclib.bary_weights([8.0, 4.0, 0.0], 9.0, bclib.params(clip_C=math.inf, eta=0.0, delta=1.0))
    np.testing.assert_allclose(w, [1.40625, -0.5625, 0.15625], rtol=1e-14)


@pytest.mark.parametrize("bad", [([], 1.0), ([1.0] * 9, 2.0), ([1.0, 1.0], 2.0), ([0.0, 2.0, 1.0], 3.0),
                                 ([math.nan], 1.0), ([1.0, 0.0], math.inf)])
def test_invalid_nodes_rejected(bclib, bad):
    with pytest.raises(bclib.BCError) as e:
        bclib.bary_weights(*bad)
    assert e.value.code == bclib.ERR_INVALID_ARG


def test_degenerate_reported(bclib):
    with pytest.raises(bclib.BCError) as e:
        bclib.bary_weights([0.5, 0.52], 0.49)
    assert e.value.code == bclib.ERR_DEGENERATE


@pytest.mark.parametrize("S,N", [(10, 3), (50, 4), (50, 5), (50, 6), (20, 4), (50, 1), (1, 3), (7, 9)])
def test_mask_bit_exact(bclib, S, N):
    assert np.array_equal(bclib.make_mask(S, N), bary.make_mask(S, N))


def test_plan_bit_exact_on_configs_and_random_masks(bclib):
    cases = []
    for cfg in synth.CONFIGS.values():
        cases.append((bary.make_mask(cfg.steps, cfg.interval), cfg.K))
    g = np.random.default_rng(12)
    for _ in range(200):
        S = int(g.integers(1, 60))
        m = (g.uniform(size=S) < 0.35).astype(np.uint8)
        m[0] = 1
        cases.append((m, int(g.integers(1, 9))))
    for mask, K in cases:
        exp = bary.plan(mask, K)
        got = bclib.plan(mask, K)
        for e, s in zip(exp, got):
            assert (bool(s.is_full), s.count, s.head) == (e.is_full, e.count, e.head)
            if not e.is_full:
                assert list(s.slots[:e.count]) == e.slots
                assert all(x == -1 for x in s.slots[e.count:])
                w = np.array(s.w[:e.count])
                assert np.max(np.abs(w - np.array(e.w))) <= _tol(w)


def test_plan_rejects_bad_masks(bclib):
    for m in ([0, 1, 1], [1, 2, 0]):
        with pytest.raises(bclib.BCError):
            bclib.plan(np.array(m, np.uint8), 2)


@pytest.mark.parametrize("sampler,S,shift", [("ddim", 10, 1.0), ("ddim", 50, 1.0), ("dpmpp2m", 20, 1.0),
                                             ("euler", 50, 1.0), ("euler", 50, 7.0), ("euler", 12, 3.0)])
def test_schedule_bit_exact(bclib, sampler, S, shift):
    tau, tm = bclib.make_schedule(sampler, S, shift)
    assert np.array_equal(tau, osm.timesteps(S))
    assert np.array_equal(tm, osm.model_time(sampler, S, shift))


def test_schedule_rejects_bad_shift(bclib):
    for shift in (-1.0, float("nan"), float("inf")):
        with pytest.raises(bclib.BCError) as e:
            bclib.make_schedule("euler", 10, shift)
        assert e.value.code == bclib.ERR_INVALID_ARG


def test_host_logic_under_address_and_ub_sanitizers(tmp_path):
    """The host plan library (plan.cpp: weights, mask, plan, schedules) built
    with -fsanitize=address,undefined and driven by random and adversarial
    arguments (tests/native/plan_fuzz.cpp); any memory or undefined-behaviour
    error aborts the run."""
    exe = tmp_path / "plan_fuzz"
    csrc = os.path.join(ROOT, "paper_2608_28670_amd", "csrc")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-I", csrc, "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "tests", "native", "plan_fuzz.cpp"), os.path.join(csrc, "plan.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "failures 0" in r.stdout


def test_kernel_symbols_demangle(bclib):
    """Every kernel symbol of the library demangles with the platform's
    demangler (c++filt): element types reach kernel templates as tags, never
    as __bf16, whose mangling (DF16b) older demanglers reject or misread —
    as profilers' kernel names then do."""
    out = subprocess.run(["nm", bclib.LIB_PATH], capture_output=True, text=True).stdout
    names = sorted({l.split()[-1] for l in out.splitlines() if "_kernel" in l and l.split()[-1].startswith("_Z")})
    assert len(names) > 50
    assert not [n for n in names if "DF16b" in n]
    dem = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True).stdout.splitlines()
    assert len(dem) == len(names)
    bad = [(n, d) for n, d in zip(names, dem) if d == n or "_Accum" in d]
    assert not bad, bad[:3]
