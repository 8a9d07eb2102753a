"""GPU parity of the forecast kernel (Eq. 13) and the cache ring, through the C ABI.

Tolerances: fp32 output, componentwise error relative to sum_j |w_j x_j| (the
condition-scaled form, since the sum can cancel) <= 1e-5; bf16 output, within
one bf16 ulp of the round-to-nearest-even of the exact value."""
import math

import numpy as np
import pytest

import synth
from oracle import bary

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def _exact(feats64, w):
    return bary.forecast(list(feats64), w), sum(abs(wj) * np.abs(f) for wj, f in zip(w, feats64))


def _bf16_ulp(x):
    a = np.abs(x).astype(np.float64)
    e = np.floor(np.log2(np.maximum(a, 1e-38)))
    return 2.0 ** (e - 7)


def check(got, exact, scale, out_dt):
    got = got.astype(np.float64)
    if out_dt == "f32":
        err = np.abs(got - exact) / np.maximum(scale, 1e-30)
        assert err.max() <= 1e-5, err.max()
    else:
        ref = synth.bf16_round(exact.astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(got - ref) <= _bf16_ulp(ref) * 1.0001 + 1e-38)


def _ring(bc, feats, dt, times):
    K = feats.shape[0]
    numel = int(np.prod(feats.shape[1:]))
    storage = torch.empty((K, numel), dtype=TDT[dt], device=DEV)
    ring = bc.CacheRing(K, storage)
    src = torch.from_numpy(feats.reshape(K, numel)).to(DEV).to(TDT[dt])
    # push oldest first so node 0 (newest) ends up last
    for j in reversed(range(K)):
        if j % 2 == 0:
            ring.push(src[j], times[j])                       # copy path
        else:
            slot = ring.next_slot()
            idx = (slot - storage.data_ptr()) // (numel * storage.element_size())
            storage[idx].copy_(src[j])
            ring.push(None, times[j])                         # zero-copy path
    return ring, storage


@pytest.mark.parametrize("K", range(1, 9))
@pytest.mark.parametrize("in_dt,out_dt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32"), ("f32", "bf16")])
@pytest.mark.parametrize("numel", [8 * 1237, 8 * 1237 + 3, 1])
def test_forecast_matches_oracle(bclib, K, in_dt, out_dt, numel):
    feats = synth.forecast_features(K, (1, numel), seed=100 + K, dtype=in_dt).reshape(K, numel)
    times = np.sort(synth.uniform(f"t{K}", (K + 1,), seed=7))
    s, t = times[1:], float(times[0])                       # newest first, query below
    try:
        w = bary.bary_weights(s, t)
    except bary.Degenerate:
        w = bary.bary_weights(s, t, bary.Params(C=math.inf))
    ring, _ = _ring(bclib, feats, in_dt, s)
    cnt, head, tn, slots = ring.state()
    assert cnt == K and list(tn) == list(s)
    out = torch.empty(numel, dtype=TDT[out_dt], device=DEV)
    bclib.bary_extrapolate(ring, w, out)
    torch.cuda.synchronize()
    exact, scale = _exact(feats.astype(np.float64), w)
    check(out.float().cpu().numpy(), exact, scale, out_dt)


def test_forecast_fewer_nodes_than_slots_and_state_errors(bclib):
    K, numel = 4, 4096
    storage = torch.zeros((K, numel), dtype=torch.float32, device=DEV)
    ring = bclib.CacheRing(K, storage)
    out = torch.empty(numel, device=DEV)
    with pytest.raises(bclib.BCError) as e:
        bclib.bary_extrapolate(ring, [1.0], out)
    assert e.value.code == bclib.ERR_STATE
    feats = synth.forecast_features(6, (1, numel), seed=3).reshape(6, numel)
    for j in range(6):                                       # wraps around: holds 5,4,3,2
        ring.push(torch.from_numpy(feats[j]).to(DEV), float(j))
    cnt, head, tn, slots = ring.state()
    assert (cnt, head, list(tn), list(slots)) == (4, 1, [5.0, 4.0, 3.0, 2.0], [1, 0, 3, 2])
    w = bary.bary_weights([5.0, 4.0], 6.0)
    bclib.bary_extrapolate(ring, w, out)
    torch.cuda.synchronize()
    exact, scale = _exact(feats[[5, 4]].astype(np.float64), w)
    check(out.cpu().numpy(), exact, scale, "f32")
    with pytest.raises(bclib.BCError):
        bclib.bary_extrapolate(ring, [0.5] * 5, out)


def test_empty_forecast_and_invalid_args(bclib):
    storage = torch.zeros((2, 16), dtype=torch.float32, device=DEV)
    ring = bclib.CacheRing(2, storage)
    ring.push(None, 0.0)
    with pytest.raises(bclib.BCError):
        bclib.bary_extrapolate(ring, [float("nan")], torch.empty(16, device=DEV))


def test_profile_times_per_launch(bclib):
    """Per-launch HIP-event durations of a kernel class, in launch order; the
    pool caps the count and collecting disables the class."""
    K, n = 2, 1 << 16
    storage = torch.randn((K, n), device=DEV)
    ring = bclib.CacheRing(K, storage)
    for j in range(K):
        ring.push(None, float(K - j))
    out = torch.empty(n, device=DEV)
    bclib.profile_enable(bclib.PROF_FORECAST, 3)
    for _ in range(5):
        bclib.bary_extrapolate(ring, [2.0, -1.0], out)
    t = bclib.profile_times(bclib.PROF_FORECAST, 8)
    assert len(t) == 3 and np.all(t > 0) and np.all(np.isfinite(t))
    bclib.bary_extrapolate(ring, [2.0, -1.0], out)
    assert len(bclib.profile_times(bclib.PROF_FORECAST, 8)) == 0
    sl = ring.state()[3]                                    # slots, newest first
    ref = 2.0 * storage[int(sl[0])] - storage[int(sl[1])]
    torch.testing.assert_close(out, ref, rtol=1e-6, atol=1e-6)
