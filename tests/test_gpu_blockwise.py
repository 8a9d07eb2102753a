"""GPU parity of blockwise mode (bc_sample_blockwise, Br = 0; Sec. 4.5, Tables
5 and 6) through the C ABI, against the oracle's sample_blockwise on the same
seeded inputs: final latents (1e-4 relative L2 for the fp32 model, 2e-2 for
bf16), and the site storage's layout [site][slot][B*T*D], read back after a
run and compared with the oracle's module outputs at the last full step."""
import numpy as np
import pytest

import synth
from oracle import bary, model as om, sampler as osm

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def rel_l2(g, r):
    return float(np.linalg.norm(np.asarray(g, np.float64) - r) / max(np.linalg.norm(r), 1e-30))


def _run(cfg, P, B, mask, labels=None, text=None):
    from paper_2608_28670_amd import loader
    dm = loader.DeviceModel(cfg, P)
    xT = synth.latents(cfg, batch=B)
    x = torch.from_numpy(np.ascontiguousarray(xT, dtype=np.float32)).to(DEV)
    tl = torch.from_numpy(labels).to(DEV) if labels is not None else None
    tt = torch.from_numpy(text).to(DEV).to(loader.torch_dtype(cfg)) if text is not None else None
    sites = dm.sample_blockwise(x, mask, labels=tl, text=tt)
    torch.cuda.synchronize()
    return dm, xT, x.cpu().numpy(), sites


CASES = {
    "tiny": (lambda: synth.CONFIGS["tiny"], 2, 1e-4),
    "dit_xl2_depth2": (lambda: synth.scaled(synth.CONFIGS["dit_xl2"], depth=2, batch=2), 2, 2e-2),
    "pixart_reduced": (lambda: synth.scaled(synth.CONFIGS["pixart"], depth=2, latent=(4, 32, 32), batch=1), 1, 2e-2),
}


@pytest.mark.parametrize("name", list(CASES))
def test_blockwise_matches_oracle(bclib, name):
    mk, B, tol = CASES[name]
    cfg = mk()
    P = synth.params(cfg)
    mask = bary.make_mask(cfg.steps, cfg.interval)
    labels = synth.labels(cfg, batch=B) if cfg.kind == "dit" and cfg.n_classes else None
    text = synth.text(cfg, batch=B) if cfg.kind == "pixart" else None
    _, xT, got, _ = _run(cfg, P, B, mask, labels, text)
    exp = osm.sample_blockwise(om.Model(cfg, P), xT.astype(np.float64), mask, cfg.K, labels=labels, text=text)
    err = rel_l2(got, exp)
    # the same run in stepwise mode differs: blockwise forecasts are not the stepwise ones
    ref = osm.sample(om.Model(cfg, P), xT.astype(np.float64), mask, cfg.K, labels=labels, text=text)
    print(f"{name}: blockwise rel-L2 {err:.2e} (stepwise oracle differs by {rel_l2(exp, ref):.2e})")
    assert err <= tol
    assert rel_l2(exp, ref) > 10 * err


def test_site_storage_layout(bclib):
    cfg = synth.CONFIGS["tiny"]
    P = synth.params(cfg)
    mask = bary.make_mask(cfg.steps, cfg.interval)
    dm, xT, _, sites = _run(cfg, P, cfg.batch, mask)
    nsites = dm.model.blockwise_sites()
    assert sites.shape == (nsites, cfg.K, cfg.batch * cfg.tokens * cfg.hidden) and nsites == 2 * cfg.depth
    # oracle module outputs at the last full step, from the latent that step started from
    M = om.Model(cfg, P)
    tr = {}
    osm.sample_blockwise(M, xT.astype(np.float64), mask, cfg.K, trace=tr)
    k = max(i for i in range(cfg.steps) if mask[i])
    head = bary.plan(mask, cfg.K)[k].head
    cond = M.condition(osm.model_time(cfg.sampler, cfg.steps)[k], cfg.batch)
    h, mods = M.embed(tr["x_in"][k]), []
    for l in range(cfg.depth):
        h = M.dit_block(l, h, M.block_mod(l, cond), None, modules=mods)
    got = sites[:, head].cpu().numpy().astype(np.float64)
    for s in range(nsites):
        e = rel_l2(got[s], mods[s].reshape(-1))
        assert e <= 1e-4, (s, e)


def test_blockwise_errors(bclib):
    from paper_2608_28670_amd import loader
    cfg = synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=256, heads=2, head_dim=128,
                       mlp=1024, latent=(16, 3, 20, 20), txt_tokens=40, batch=1)
    dm = loader.DeviceModel(cfg, synth.params(cfg))
    with pytest.raises(bclib.BCError) as e:
        dm.model.blockwise_sites()
    assert e.value.code == bclib.ERR_UNSUPPORTED
    tiny = synth.CONFIGS["tiny"]
    dt = loader.DeviceModel(tiny, synth.params(tiny))
    x = torch.zeros((tiny.batch,) + tuple(tiny.latent), dtype=torch.float32, device=DEV)
    mask = bary.make_mask(tiny.steps, tiny.interval)
    ws, _ = dt.buffers(tiny.batch, tiny.K, tiny.steps)
    store = torch.empty(2 * tiny.depth * tiny.K * tiny.batch * tiny.tokens * tiny.hidden + 4, dtype=torch.float32,
                        device=DEV)
    with pytest.raises(bclib.BCError) as e:     # storage not 16-byte aligned
        bclib.sample_blockwise(dt.model, tiny.batch, tiny.sampler, mask, tiny.K, store[1:], x, ws)
    assert e.value.code == bclib.ERR_INVALID_ARG
    with pytest.raises(bclib.BCError) as e:     # K outside 1..8
        bclib.sample_blockwise(dt.model, tiny.batch, tiny.sampler, mask, 9, store, x, ws)
    assert e.value.code == bclib.ERR_INVALID_ARG
    with pytest.raises(bclib.BCError) as e:     # storage one slot short
        short = store[:2 * tiny.depth * (tiny.K - 1) * tiny.batch * tiny.tokens * tiny.hidden]
        bclib.sample_blockwise(dt.model, tiny.batch, tiny.sampler, mask, tiny.K, short, x, ws)
    assert e.value.code == bclib.ERR_INVALID_ARG
