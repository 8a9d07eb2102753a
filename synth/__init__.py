"""Seeded synthetic inputs for the BaryCache hot path.

This module is shared by the CPU oracle's tests and by the GPU path (tests,
smoke run, benchmark).  It holds none of the method's arithmetic: only
counter-based random draws keyed by tensor name, round-to-nearest-even
conversion of those draws to bfloat16 values, and the shape tables of the
synthetic workloads (tensor names and sizes).

Every tensor is drawn from its own Philox stream whose 128-bit key is a hash
of (seed, tensor name), so any tensor can be regenerated alone, in any order,
on any machine.  The default seed is the one the paper states for all of its
runs (Experimental Setup section).
"""
from __future__ import annotations

import dataclasses
import hashlib
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Iterable, List, Optional, Tuple

import numpy as np

SEED = 2026


def _key(seed: int, name: str) -> int:
    h = hashlib.sha256(f"{seed}/{name}".encode()).digest()
    return int.from_bytes(h[:16], "little")


def rng(name: str, seed: int = SEED) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(key=_key(seed, name)))


def normal(name: str, shape, scale: float = 1.0, seed: int = SEED) -> np.ndarray:
    """N(0,1)*scale draws as float32, from the stream keyed by `name`."""
    a = rng(name, seed).standard_normal(size=tuple(shape), dtype=np.float32)
    if scale != 1.0:
        a *= np.float32(scale)
    return a


def uniform(name: str, shape, lo: float = 0.0, hi: float = 1.0, seed: int = SEED) -> np.ndarray:
    """Uniform [lo, hi) draws as float64."""
    return rng(name, seed).uniform(lo, hi, size=tuple(shape))


def integers(name: str, shape, hi: int, seed: int = SEED) -> np.ndarray:
    return rng(name, seed).integers(0, hi, size=tuple(shape), dtype=np.int64)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32.

    Finite inputs only (the draws here are finite)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    r = (u + bias) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) of the RNE rounding of float32 values."""
    return (bf16_round(a).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# ---------------------------------------------------------------------------
# Workload shapes
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class ModelConfig:
    """Shape of a synthetic DiT-family model and of one sampling job."""
    name: str
    kind: str              # "dit" | "pixart" | "mmdit" (dual- then single-stream)
    depth: int             # blocks (dit/pixart); for mmdit: dual-stream blocks
    depth_single: int      # mmdit: single-stream blocks (0 otherwise)
    hidden: int            # D
    heads: int
    head_dim: int
    mlp: int               # MLP hidden width
    in_ch: int             # latent channels
    out_ch: int            # model output channels
    patch: Tuple[int, ...]  # (p,) for images, (pt, p, p) would be video; here spatial patch p
    latent: Tuple[int, ...]  # (C, H, W) or (C, F, H, W)
    batch: int
    steps: int
    sampler: str           # "ddim" | "dpmpp2m" | "euler"
    K: int                 # barycentric nodes (history length)
    interval: int          # one full step every `interval` steps
    dtype: str             # "f32" | "bf16"
    n_classes: int = 0     # class-conditional: table has n_classes+1 rows
    ctx_tokens: int = 0    # pixart cross-attention context length
    ctx_dim: int = 0       # pixart raw text width
    txt_tokens: int = 0    # mmdit text stream tokens
    qk_norm: bool = False  # mmdit: RMSNorm (learned scale) on each head's queries and keys
    rope_theta: float = 0.0  # mmdit: 3D rotary embedding of the image tokens' queries and keys (0: none)
    flow_shift: float = 1.0  # euler: time shift of the flow-matching schedule (1: none)
    param_scale: float = 0.02
    latent_scale: float = 1.0
    freq_dim: int = 256

    @property
    def p(self) -> int:
        return self.patch[0]

    @property
    def tokens(self) -> int:
        """Image (latent) tokens per sample."""
        if len(self.latent) == 3:
            _, h, w = self.latent
            return (h // self.p) * (w // self.p)
        _, f, h, w = self.latent
        return f * (h // self.p) * (w // self.p)

    @property
    def patch_dim(self) -> int:
        return self.in_ch * self.p * self.p

    @property
    def out_patch_dim(self) -> int:
        return self.out_ch * self.p * self.p


# The synthetic workloads.  Sizes follow the models the paper evaluates
# (Experimental Setup section): a tiny fp32 DiT for exact checks, a
# DiT-XL/2-shaped class-conditional model, a PixArt-shaped text-to-image model
# and a HunyuanVideo-shaped text-to-video model.
CONFIGS: Dict[str, ModelConfig] = {
    "tiny": ModelConfig(
        name="tiny", kind="dit", depth=2, depth_single=0, hidden=128, heads=4, head_dim=32,
        mlp=512, in_ch=4, out_ch=4, patch=(1,), latent=(4, 8, 8), batch=2, steps=10,
        sampler="ddim", K=3, interval=3, dtype="f32", latent_scale=0.02),
    "dit_xl2": ModelConfig(
        name="dit_xl2", kind="dit", depth=28, depth_single=0, hidden=1152, heads=16, head_dim=72,
        mlp=4608, in_ch=4, out_ch=8, patch=(2,), latent=(4, 32, 32), batch=16, steps=50,
        sampler="ddim", K=3, interval=4, dtype="bf16", n_classes=1000),
    "pixart": ModelConfig(
        name="pixart", kind="pixart", depth=28, depth_single=0, hidden=1152, heads=16, head_dim=72,
        mlp=4608, in_ch=4, out_ch=8, patch=(2,), latent=(4, 128, 128), batch=4, steps=20,
        sampler="dpmpp2m", K=4, interval=4, dtype="bf16", ctx_tokens=120, ctx_dim=4096),
    "hunyuan": ModelConfig(
        name="hunyuan", kind="mmdit", depth=20, depth_single=40, hidden=3072, heads=24, head_dim=128,
        mlp=12288, in_ch=16, out_ch=16, patch=(2,), latent=(16, 9, 60, 106), batch=1, steps=50,
        sampler="euler", K=3, interval=5, dtype="bf16", txt_tokens=256, qk_norm=True, rope_theta=256.0,
        flow_shift=7.0),
}


def scaled(cfg: ModelConfig, **kw) -> ModelConfig:
    """A copy of `cfg` with some fields replaced (reduced depth or batch for tests)."""
    return dataclasses.replace(cfg, **kw)


def param_shapes(cfg: ModelConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    """Names and shapes of every parameter of the synthetic model.

    Linear weights are [out, in] (row-major, input dimension contiguous)."""
    D, F, fd = cfg.hidden, cfg.mlp, cfg.freq_dim
    out: List[Tuple[str, Tuple[int, ...]]] = [
        ("t_w1", (D, fd)), ("t_b1", (D,)), ("t_w2", (D, D)), ("t_b2", (D,)),
        ("patch_w", (D, cfg.patch_dim)), ("patch_b", (D,)), ("pos", (cfg.tokens, D)),
    ]
    if cfg.n_classes:
        out.append(("y_table", (cfg.n_classes + 1, D)))
    if cfg.kind in ("dit", "pixart"):
        if cfg.kind == "pixart":
            out += [("t6_w", (6 * D, D)), ("t6_b", (6 * D,)),
                    ("cap_w1", (D, cfg.ctx_dim)), ("cap_b1", (D,)),
                    ("cap_w2", (D, D)), ("cap_b2", (D,))]
        for l in range(cfg.depth):
            p = f"blocks.{l}."
            if cfg.kind == "dit":
                out += [(p + "w_mod", (6 * D, D)), (p + "b_mod", (6 * D,))]
            else:
                out += [(p + "table", (6, D))]
            out += [(p + "w_qkv", (3 * D, D)), (p + "b_qkv", (3 * D,)),
                    (p + "w_o", (D, D)), (p + "b_o", (D,))]
            if cfg.kind == "pixart":
                out += [(p + "wx_q", (D, D)), (p + "bx_q", (D,)),
                        (p + "wx_kv", (2 * D, D)), (p + "bx_kv", (2 * D,)),
                        (p + "wx_o", (D, D)), (p + "bx_o", (D,))]
            out += [(p + "w_fc1", (F, D)), (p + "b_fc1", (F,)),
                    (p + "w_fc2", (D, F)), (p + "b_fc2", (D,))]
        if cfg.kind == "dit":
            out += [("final_w_mod", (2 * D, D)), ("final_b_mod", (2 * D,))]
        else:
            out += [("final_table", (2, D))]
    else:  # mmdit
        out += [("txt_w", (D, D)), ("txt_b", (D,))]
        for l in range(cfg.depth):
            p = f"dual.{l}."
            for s in ("img", "txt"):
                q = p + s + "."
                out += [(q + "w_mod", (6 * D, D)), (q + "b_mod", (6 * D,)),
                        (q + "w_qkv", (3 * D, D)), (q + "b_qkv", (3 * D,)),
                        (q + "w_o", (D, D)), (q + "b_o", (D,)),
                        (q + "w_fc1", (F, D)), (q + "b_fc1", (F,)),
                        (q + "w_fc2", (D, F)), (q + "b_fc2", (D,))]
                if cfg.qk_norm:
                    out += [(q + "q_norm", (cfg.head_dim,)), (q + "k_norm", (cfg.head_dim,))]
        for l in range(cfg.depth_single):
            p = f"single.{l}."
            out += [(p + "w_mod", (3 * D, D)), (p + "b_mod", (3 * D,)),
                    (p + "w_1", (3 * D + F, D)), (p + "b_1", (3 * D + F,)),
                    (p + "w_2", (D, D + F)), (p + "b_2", (D,))]
            if cfg.qk_norm:
                out += [(p + "q_norm", (cfg.head_dim,)), (p + "k_norm", (cfg.head_dim,))]
        out += [("final_w_mod", (2 * D, D)), ("final_b_mod", (2 * D,))]
    out += [("final_w", (cfg.out_patch_dim, D)), ("final_b", (cfg.out_patch_dim,))]
    return out


def param(cfg: ModelConfig, name: str, shape, seed: int = SEED) -> np.ndarray:
    """One parameter tensor: N(0,1)*scale (norm scales: 1 + N(0,1)*scale),
    rounded to bf16 values for bf16 models."""
    a = normal(f"{cfg.name}/{name}", shape, cfg.param_scale, seed)
    if name.endswith("_norm"):
        a = (a + 1.0).astype(np.float32)
    return bf16_round(a) if cfg.dtype == "bf16" else a


def params(cfg: ModelConfig, seed: int = SEED, names: Optional[Iterable[str]] = None,
           threads: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Every parameter (or the named subset) as float32 arrays, drawn in parallel."""
    shapes = param_shapes(cfg)
    if names is not None:
        want = set(names)
        shapes = [(n, s) for n, s in shapes if n in want]
    nt = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(nt) as ex:
        arrs = list(ex.map(lambda ns: param(cfg, ns[0], ns[1], seed), shapes))
    return {n: a for (n, _), a in zip(shapes, arrs)}


def latents(cfg: ModelConfig, seed: int = SEED, batch: Optional[int] = None) -> np.ndarray:
    """Initial noise x_T, float32 [B, *latent]."""
    B = batch or cfg.batch
    return normal(f"{cfg.name}/x_T", (B,) + tuple(cfg.latent), cfg.latent_scale, seed)


def labels(cfg: ModelConfig, seed: int = SEED, batch: Optional[int] = None) -> np.ndarray:
    """Class labels, uniform over the real classes (int64 [B])."""
    B = batch or cfg.batch
    return integers(f"{cfg.name}/labels", (B,), cfg.n_classes, seed)


def text(cfg: ModelConfig, seed: int = SEED, batch: Optional[int] = None) -> np.ndarray:
    """Synthetic text-encoder output: pixart [B, ctx_tokens, ctx_dim], mmdit [B, txt_tokens, D].

    Values N(0,1), rounded to bf16 values for bf16 models."""
    B = batch or cfg.batch
    if cfg.kind == "pixart":
        shape = (B, cfg.ctx_tokens, cfg.ctx_dim)
    else:
        shape = (B, cfg.txt_tokens, cfg.hidden)
    a = normal(f"{cfg.name}/text", shape, 1.0, seed)
    return bf16_round(a) if cfg.dtype == "bf16" else a


# ---------------------------------------------------------------------------
# Forecast microbenchmark inputs: K cached feature tensors plus node times
# ---------------------------------------------------------------------------

FORECAST_SHAPE = (8, 16384, 3072)


def forecast_features(K: int, shape=FORECAST_SHAPE, seed: int = SEED, dtype: str = "f32",
                      threads: Optional[int] = None) -> np.ndarray:
    """[K, *shape] N(0,1) features (bf16-rounded values when dtype == 'bf16').

    Slot j, leading index i is drawn from its own stream, so the large
    microbenchmark tensors are generated in parallel."""
    tag = f"forecast/feat/{'x'.join(map(str, shape))}"
    out = np.empty((K,) + tuple(shape), dtype=np.float32)
    jobs = [(j, i) for j in range(K) for i in range(shape[0])]

    def fill(ji):
        j, i = ji
        a = normal(f"{tag}/{j}/{i}", shape[1:], 1.0, seed)
        out[j, i] = bf16_round(a) if dtype == "bf16" else a

    nt = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(nt) as ex:
        list(ex.map(fill, jobs))
    return out


def forecast_times(K: int, seed: int = SEED) -> Tuple[np.ndarray, float]:
    """K node times and a query time in [0, 1], as a sampler running from
    t = 1 down to 0 sees them: K+1 uniform draws sorted decreasingly; the first
    K are the cached times and the last one is the query, below them all.  The
    nodes are returned newest first, i.e. nearest to the query first."""
    u = np.sort(uniform(f"forecast/times/K{K}", (K + 1,), seed=seed))[::-1]
    return np.ascontiguousarray(u[:K][::-1]), float(u[K])
