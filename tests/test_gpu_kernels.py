"""GPU parity of the building blocks through the C ABI: MFMA linear layers with
their fused epilogues, and attention, against the oracle's plain definitions
on the same (bf16-rounded where bf16) inputs."""
import numpy as np
import pytest

import synth
from oracle import model as om

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def rel_l2(g, r):
    return float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30))


def _inputs(name, shape, dt, scale=1.0):
    a = synth.normal(name, shape, scale)
    return synth.bf16_round(a) if dt == "bf16" else a


def _dev(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(TDT[dt])


@pytest.mark.parametrize("dt", ["bf16", "f32"])
# Beyond the small and model shapes, four bf16 shapes reach each multi-round tile
# of the wide kernel with a ragged row tail: 256 x 288 with a ragged column tile
# (4100 x 4616), 256 x 256 (4100 x 4352), 128 x 432 (4000 x 3456) and 128 x 128
# (4000 x 2304).
@pytest.mark.parametrize("M,N,K", [(300, 200, 136), (128, 128, 64), (1, 16, 8), (517, 384, 1152),
                                   (4096, 1152, 1152), (4100, 4612, 1152), (130, 260, 192), (1000, 1160, 256),
                                   (4100, 4616, 64), (4100, 4352, 128), (4000, 3456, 64), (4000, 2304, 64)])
@pytest.mark.parametrize("epi", ["bias", "gelu", "gate"])
def test_linear(bclib, dt, M, N, K, epi):
    if dt == "f32" and M * N * K > 1e8:
        pytest.skip("fp32 path is for the small model")
    A = _inputs(f"A{M}{N}{K}", (M, K), dt)
    W = _inputs(f"W{M}{N}{K}", (N, K), dt, 0.05)
    b = _inputs(f"b{M}{N}{K}", (N,), dt, 0.1)
    y = om.linear(A.astype(np.float64), W.astype(np.float64), b.astype(np.float64))
    tA, tW, tb = _dev(A, dt), _dev(W, dt), _dev(b, dt)
    if epi == "gate":
        rpg = max(1, M // 3)
        G = synth.normal(f"g{M}", ((M + rpg - 1) // rpg, N), 0.5)
        R = synth.normal(f"r{M}", (M, N), 1.0)
        exp = R.astype(np.float64) + np.repeat(G, rpg, axis=0)[:M] * y
        out = torch.from_numpy(R).to(DEV)
        bclib.linear(tA, tW, tb, out, bclib.EPI_GATE_RES, res=out, gate=torch.from_numpy(G).to(DEV),
                     rows_per_gate=rpg)
        tol = 1e-5
    else:
        exp = om.gelu_tanh(y) if epi == "gelu" else y
        out = torch.empty((M, N), dtype=TDT[dt], device=DEV)
        bclib.linear(tA, tW, tb, out, bclib.EPI_BIAS_GELU if epi == "gelu" else bclib.EPI_BIAS)
        tol = 5e-3 if dt == "bf16" else 1e-5
    torch.cuda.synchronize()
    err = rel_l2(out.float().cpu().numpy().astype(np.float64), exp)
    assert err <= tol, err


def test_linear_rejects_bad_k(bclib):
    A = torch.zeros((4, 12), dtype=torch.bfloat16, device=DEV)
    W = torch.zeros((16, 12), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(bclib.BCError) as e:
        bclib.linear(A, W, None, torch.empty((4, 16), dtype=torch.bfloat16, device=DEV))
    assert e.value.code == bclib.ERR_UNSUPPORTED


@pytest.mark.parametrize("dt,B,H,Tq,Tk,d", [
    ("bf16", 2, 3, 200, 200, 72), ("bf16", 1, 2, 100, 37, 128), ("bf16", 2, 2, 64, 64, 32),
    ("bf16", 1, 1, 130, 257, 64), ("bf16", 1, 1, 1, 1, 72), ("bf16", 16, 16, 256, 256, 72),
    ("bf16", 1, 2, 1100, 700, 72), ("bf16", 2, 1, 600, 1030, 32), ("bf16", 1, 2, 520, 333, 128),
    # enough (sample, head) pairs for the 256- and 512-query workgroups
    ("bf16", 8, 32, 300, 300, 72), ("bf16", 8, 32, 300, 270, 64), ("bf16", 4, 32, 300, 333, 128),
    # resident key tiles with 32 queries per wave (short key sequences, large grids)
    ("bf16", 8, 32, 300, 120, 72), ("bf16", 8, 32, 300, 200, 128), ("bf16", 8, 32, 260, 256, 32),
    ("f32", 2, 4, 64, 64, 32), ("f32", 1, 2, 77, 131, 64)])
def test_attention(bclib, dt, B, H, Tq, Tk, d):
    q = _inputs(f"q{Tq}{d}", (B, Tq, H, d), dt)
    k = _inputs(f"k{Tk}{d}", (B, Tk, H, d), dt)
    v = _inputs(f"v{Tk}{d}", (B, Tk, H, d), dt)
    exp = om.attention(*(a.astype(np.float64).transpose(0, 2, 1, 3) for a in (q, k, v))).transpose(0, 2, 1, 3)
    out = torch.empty((B, Tq, H, d), dtype=TDT[dt], device=DEV)
    bclib.attention(_dev(q, dt), _dev(k, dt), _dev(v, dt), out)
    torch.cuda.synchronize()
    err = rel_l2(out.float().cpu().numpy().astype(np.float64), exp)
    assert err <= (1e-2 if dt == "bf16" else 1e-5), err


# Pre-scaled queries (the form the blocks' projections write): every key-loop
# variant, i.e. the resident loop, and the streaming loop with 16, 32 (4-wave
# workgroups at d = 128, 8-wave otherwise) and 64 queries per wave; at d = 128
# the last key tile holds 13 keys (333) or 54 (310).
@pytest.mark.parametrize("B,H,Tq,Tk,d", [
    (16, 16, 256, 256, 72), (1, 2, 100, 37, 128), (1, 2, 1100, 700, 72), (1, 2, 520, 333, 128),
    (2, 1, 600, 1030, 32), (4, 16, 300, 300, 72), (4, 32, 300, 333, 128), (4, 32, 300, 310, 128),
    (8, 32, 300, 300, 72), (8, 32, 300, 270, 64), (8, 32, 300, 120, 72), (8, 32, 300, 200, 128),
    (1, 1, 1, 1, 72)])
def test_attention_prescaled(bclib, B, H, Tq, Tk, d):
    q = _inputs(f"q{Tq}{d}", (B, Tq, H, d), "bf16")
    k = _inputs(f"k{Tk}{d}", (B, Tk, H, d), "bf16")
    v = _inputs(f"v{Tk}{d}", (B, Tk, H, d), "bf16")
    # the producer's rounding: q * log2(e) / sqrt(d) in fp32, rounded to bf16
    c = np.float32(1.4426950408889634) / np.sqrt(np.float32(d))
    qs = synth.bf16_round((q.astype(np.float32) * c).astype(np.float32))
    # softmax(q k^T / sqrt(d)) with the queries the stored values stand for
    qeff = qs.astype(np.float64) / float(c)
    exp = om.attention(*(a.astype(np.float64).transpose(0, 2, 1, 3) for a in (qeff, k, v))).transpose(0, 2, 1, 3)
    out = torch.empty((B, Tq, H, d), dtype=torch.bfloat16, device=DEV)
    bclib.attention(_dev(qs, "bf16"), _dev(k, "bf16"), _dev(v, "bf16"), out, prescaled=True)
    torch.cuda.synchronize()
    err = rel_l2(out.float().cpu().numpy().astype(np.float64), exp)
    assert err <= 1e-2, err


# Output rows that are not 8-byte aligned take the per-element stores.
@pytest.mark.parametrize("B,H,Tq,Tk,d", [(2, 3, 200, 200, 72), (1, 2, 520, 333, 128)])
def test_attention_unaligned_output(bclib, B, H, Tq, Tk, d):
    q = _inputs(f"q{Tq}{d}", (B, Tq, H, d), "bf16")
    k = _inputs(f"k{Tk}{d}", (B, Tk, H, d), "bf16")
    v = _inputs(f"v{Tk}{d}", (B, Tk, H, d), "bf16")
    exp = om.attention(*(a.astype(np.float64).transpose(0, 2, 1, 3) for a in (q, k, v))).transpose(0, 2, 1, 3)
    n = B * Tq * H * d
    buf = torch.zeros(n + 2, dtype=torch.bfloat16, device=DEV)
    out = buf[2:].view(B, Tq, H, d)     # 4 bytes past an aligned start
    assert out.data_ptr() % 8 == 4
    bclib.attention(_dev(q, "bf16"), _dev(k, "bf16"), _dev(v, "bf16"), out)
    torch.cuda.synchronize()
    err = rel_l2(out.float().cpu().numpy().astype(np.float64), exp)
    assert err <= 1e-2, err
    assert float(buf[:2].abs().sum()) == 0.0     # nothing written before the output


def test_attention_prescaled_rejects_fp32(bclib):
    z = torch.zeros((1, 4, 1, 32), dtype=torch.float32, device=DEV)
    with pytest.raises(bclib.BCError) as e:
        bclib.attention(z, z, z, torch.empty_like(z), prescaled=True)
    assert e.value.code == bclib.ERR_UNSUPPORTED


def test_attention_rejects_unsupported_head_dim(bclib):
    z = torch.zeros((1, 4, 1, 40), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(bclib.BCError) as e:
        bclib.attention(z, z, z, torch.empty_like(z))
    assert e.value.code == bclib.ERR_UNSUPPORTED
