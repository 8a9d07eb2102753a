"""GPU parity of the adaptive schedule (bc_sample_adaptive, Sec. 4.5, Table 5)
through the C ABI, against the oracle's sample_adaptive on the same seeded
inputs.

The realised mask is integer output: it must equal the oracle's.  The
thresholds are chosen so that every accumulated sum the oracle compares with
the threshold is at least 4 % away from it (the decisions cannot flip within
the tolerance of the bf16 changes).  Changes are gated per step (1e-5 relative
for the fp32 model, 2e-2 for bf16), final latents like bc_sample's (1e-4 fp32,
2e-2 bf16).  Independently of the oracle, an adaptive run must equal bc_sample
bit for bit under the mask it realised, and that mask must be the one the rule
gives for the changes the run reported."""
import math

import numpy as np
import pytest

import synth
from oracle import model as om, sampler as osm

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def rel_l2(g, r):
    return float(np.linalg.norm(np.asarray(g, np.float64) - r) / max(np.linalg.norm(r), 1e-30))


def _inputs(cfg, B):
    labels = synth.labels(cfg, batch=B) if cfg.kind == "dit" and cfg.n_classes else None
    text = synth.text(cfg, batch=B) if cfg.kind != "dit" else None
    return synth.latents(cfg, batch=B), labels, text


def _gpu(cfg, P, B, ell, dm=None):
    from paper_2608_28670_amd import loader
    dm = dm or loader.DeviceModel(cfg, P)
    xT, labels, text = _inputs(cfg, B)
    x = torch.from_numpy(np.ascontiguousarray(xT, dtype=np.float32)).to(DEV)
    tl = torch.from_numpy(labels).to(DEV) if labels is not None else None
    tt = torch.from_numpy(text).to(DEV).to(loader.torch_dtype(cfg)) if text is not None else None
    _, mask, change = dm.sample_adaptive(x, cfg.steps, ell, labels=tl, text=tt)
    torch.cuda.synchronize()
    return dm, xT, x, mask, change, tl, tt


def _mm_cfg():
    return synth.scaled(synth.CONFIGS["hunyuan"], depth=1, depth_single=1, hidden=256, heads=2, head_dim=128,
                        mlp=1024, latent=(16, 3, 20, 20), txt_tokens=40, batch=2, steps=12)


CASES = {
    "tiny": (lambda: synth.CONFIGS["tiny"], 0.3, 1e-5, 1e-4),
    "dit_xl2_depth2": (lambda: synth.scaled(synth.CONFIGS["dit_xl2"], depth=2, batch=2), 0.12, 2e-2, 2e-2),
    "pixart_reduced": (lambda: synth.scaled(synth.CONFIGS["pixart"], depth=2, latent=(4, 32, 32), batch=1), 0.09,
                       2e-2, 2e-2),
    "mmdit_reduced": (_mm_cfg, 0.05, 2e-2, 2e-2),
}


@pytest.mark.parametrize("name", list(CASES))
def test_adaptive_matches_oracle(bclib, name):
    mk, ell, tol_change, tol_x = CASES[name]
    cfg = mk()
    B = cfg.batch
    P = synth.params(cfg)
    _, xT, x, mask, change, _, _ = _gpu(cfg, P, B, ell)
    _, labels, text = _inputs(cfg, B)
    tr = {}
    exp_x, exp_mask, exp_change = osm.sample_adaptive(om.Model(cfg, P), xT.astype(np.float64), cfg.steps, ell,
                                                      cfg.K, labels=labels, text=text, trace=tr)
    acc = np.array(tr["acc"][1:-1])
    assert np.min(np.abs(acc - ell)) >= 0.04 * ell        # the case keeps its decisions away from ell
    assert 2 < sum(exp_mask) < cfg.steps
    print(f"{name}: ell {ell}, full steps {int(mask.sum())} (oracle {sum(exp_mask)})")
    assert list(mask) == exp_mask
    assert change[0] == 0.0
    err_c = np.abs(change[1:] - np.array(exp_change[1:])) / np.array(exp_change[1:])
    err_x = rel_l2(x.cpu().numpy(), exp_x)
    print(f"  max change rel err {err_c.max():.2e}, final latents rel-L2 {err_x:.2e}")
    assert err_c.max() <= tol_change
    assert err_x <= tol_x


@pytest.mark.parametrize("name", ["dit_xl2_depth2", "mmdit_reduced"])
def test_adaptive_is_the_fixed_loop_under_its_mask(bclib, name):
    mk, ell, _, _ = CASES[name]
    cfg = mk()
    dm, xT, x, mask, change, tl, tt = _gpu(cfg, synth.params(cfg), cfg.batch, ell)
    assert list(mask) == osm.adaptive_mask(change, ell)
    x2 = torch.from_numpy(np.ascontiguousarray(xT, dtype=np.float32)).to(DEV)
    dm.sample(x2, mask, labels=tl, text=tt)
    torch.cuda.synchronize()
    assert torch.equal(x, x2)


def test_adaptive_threshold_limits(bclib):
    cfg = synth.scaled(synth.CONFIGS["dit_xl2"], depth=2, batch=2, steps=12)
    dm, xT, x, mask, change, tl, tt = _gpu(cfg, synth.params(cfg), 2, 0.0)
    assert list(mask) == [1] * cfg.steps and np.all(change[1:] > 0)
    x2 = torch.from_numpy(np.ascontiguousarray(xT, dtype=np.float32)).to(DEV)
    dm.sample(x2, mask, labels=tl, text=tt)
    torch.cuda.synchronize()
    assert torch.equal(x, x2)
    _, _, _, mask, _, _, _ = _gpu(cfg, None, 2, math.inf, dm=dm)
    assert list(mask) == [1] + [0] * (cfg.steps - 2) + [1]


def test_adaptive_errors(bclib):
    from paper_2608_28670_amd import loader
    cfg = synth.CONFIGS["tiny"]
    dm = loader.DeviceModel(cfg, synth.params(cfg))
    x = torch.zeros((cfg.batch,) + tuple(cfg.latent), dtype=torch.float32, device=DEV)
    for ell in (float("nan"), -0.5):
        with pytest.raises(bclib.BCError) as e:
            dm.sample_adaptive(x, cfg.steps, ell)
        assert e.value.code == bclib.ERR_INVALID_ARG
    ws, ring = dm.buffers(cfg.batch, cfg.K, cfg.steps)     # bc_sample's workspace is too small here
    assert ws.numel() < dm.model.adaptive_workspace_size(cfg.batch, cfg.steps)
    with pytest.raises(bclib.BCError) as e:
        bclib.sample_adaptive(dm.model, cfg.batch, cfg.sampler, cfg.steps, 0.3, cfg.K, ring, x, ws)
    assert e.value.code == bclib.ERR_INVALID_ARG
