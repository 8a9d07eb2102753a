"""The sampling loop captured as a HIP graph and replayed (bc_sample_graph_*),
through the C ABI.

Every replay must reproduce the eager bc_sample run bit for bit (same kernels,
same inputs, same order); the tiny fp32 model is also held to the oracle.
Replays are interleaved with the program's own eager work (refilling x_T, an
eager run on the same ring and workspace) and synchronisations."""
import numpy as np
import pytest

import synth
from oracle import bary, model as om, sampler as osm

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _setup(cfg, B, labels=None, text=None):
    from paper_2608_28670_amd import loader
    P = synth.params(cfg)
    dm = loader.DeviceModel(cfg, P)
    xT = torch.from_numpy(np.ascontiguousarray(synth.latents(cfg, batch=B), dtype=np.float32)).to(DEV)
    tl = torch.from_numpy(labels).to(DEV) if labels is not None else None
    tt = torch.from_numpy(text).to(DEV).to(loader.torch_dtype(cfg)) if text is not None else None
    return P, dm, xT, tl, tt


def _replays_match_eager(dm, xT, mask, tl, tt, replays=3):
    x = xT.clone()
    ring = dm.sample(x, mask, labels=tl, text=tt)
    torch.cuda.synchronize()
    eager, eager_state = x.clone(), ring.state()
    xg = torch.empty_like(xT)
    ring.reset()
    g = dm.sample_graph(xg, mask, labels=tl, text=tt)
    assert ring.state()[0] == 0                       # capturing ran nothing
    for r in range(replays):
        xg.copy_(xT)
        g.launch()
        torch.cuda.synchronize()
        assert torch.equal(xg, eager), f"replay {r}"
        st = ring.state()
        assert st[0] == eager_state[0] and st[1] == eager_state[1]
        assert np.array_equal(st[2], eager_state[2]) and np.array_equal(st[3], eager_state[3])
        x2 = xT.clone()                               # eager work on the same ring and workspace
        dm.sample(x2, mask, labels=tl, text=tt)
        torch.cuda.synchronize()
        assert torch.equal(x2, eager)
    del g
    return eager


def test_graph_tiny_fp32(bclib):
    cfg = synth.CONFIGS["tiny"]
    P, dm, xT, tl, tt = _setup(cfg, cfg.batch)
    mask = bary.make_mask(cfg.steps, cfg.interval)
    got = _replays_match_eager(dm, xT, mask, tl, tt).cpu().numpy().astype(np.float64)
    exp = osm.sample(om.Model(cfg, P), xT.cpu().numpy().astype(np.float64), mask, cfg.K)
    assert np.linalg.norm(got - exp) / np.linalg.norm(exp) <= 1e-4


def test_graph_dit_xl2_reduced_depth(bclib):
    cfg = synth.scaled(synth.CONFIGS["dit_xl2"], depth=2, batch=2)
    labels = synth.labels(cfg, batch=2)
    _, dm, xT, tl, tt = _setup(cfg, 2, labels=labels)
    _replays_match_eager(dm, xT, bary.make_mask(cfg.steps, cfg.interval), tl, tt)


def test_graph_pixart_reduced(bclib):
    cfg = synth.scaled(synth.CONFIGS["pixart"], depth=2, latent=(4, 32, 32), batch=1)
    text = synth.text(cfg, batch=1)
    _, dm, xT, tl, tt = _setup(cfg, 1, text=text)
    _replays_match_eager(dm, xT, bary.make_mask(cfg.steps, cfg.interval), tl, tt, replays=2)


def test_graph_errors(bclib):
    cfg = synth.CONFIGS["tiny"]
    _, dm, xT, tl, tt = _setup(cfg, cfg.batch)
    mask = bary.make_mask(cfg.steps, cfg.interval)
    ws, ring = dm.buffers(cfg.batch, cfg.K, len(mask))
    x = xT.clone()
    null = torch.cuda.default_stream()
    with pytest.raises(bclib.BCError) as e:        # the null stream cannot capture
        bclib.SampleGraph(dm.model, cfg.batch, cfg.sampler, mask, cfg.K, ring, x, ws, stream=null)
    assert e.value.code == bclib.ERR_INVALID_ARG
    bclib.profile_enable(bclib.PROF_GEMM_BIAS, 4)
    with pytest.raises(bclib.BCError) as e:        # timing on
        bclib.SampleGraph(dm.model, cfg.batch, cfg.sampler, mask, cfg.K, ring, x, ws)
    assert e.value.code == bclib.ERR_STATE
    bclib.profile_times(bclib.PROF_GEMM_BIAS, 4)
    bad = np.zeros(cfg.steps, np.uint8)             # mask[0] must be 1: bc_sample's own check
    with pytest.raises(bclib.BCError) as e:
        bclib.SampleGraph(dm.model, cfg.batch, cfg.sampler, bad, cfg.K, ring, x, ws)
    assert e.value.code == bclib.ERR_INVALID_ARG
    # A failed capture leaves the stream usable: an eager run still matches a fresh one.
    x1, x2 = xT.clone(), xT.clone()
    dm.sample(x1, mask)
    dm.sample(x2, mask)
    torch.cuda.synchronize()
    assert torch.equal(x1, x2)
