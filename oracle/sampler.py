"""Oracle: noise schedules, sampler updates and the BaryCache sampling loop.

TEST INFRASTRUCTURE ONLY (tests, smoke check and the benchmark's CPU baseline
import it).  Plain numpy in fp64.  Shares no code with the HIP library.

The paper states the DDPM forward process and reverse mean (Sec. 3.1, Eqs. 1-3)
and names the samplers it runs: DDIM for class- and text-to-image, Euler for
text-to-video, 50 steps (Sec. 4.1).  The precise samplers below are readings:
  * linear beta schedule 1e-4 .. 0.02 over 1000 training steps; alpha_bar is
    the running product of (1 - beta) (Eq. 3's definition);
  * "trailing" integer timesteps tau_k = 999 - floor(1000 k / S);
  * DDIM with eta = 0 (deterministic); the last step maps to alpha_bar = 1;
  * DPM-Solver++(2M) in the data-prediction form with the same timesteps;
  * Euler on the flow-matching ODE with sigma_k = 1 - k/S, model time 1000 sigma.
The loop itself is Sec. 3.3: on a full step run the stack and store its output
in the cache; otherwise forecast it from the cache with Eq. 13; then the final
layer and the sampler update.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import bary
from .model import Model

T_TRAIN = 1000


def alpha_bar_table(n: int = T_TRAIN) -> np.ndarray:
    beta = 1e-4 + (0.02 - 1e-4) * np.arange(n, dtype=np.float64) / (n - 1)
    return np.cumprod(1.0 - beta)


def timesteps(S: int) -> np.ndarray:
    """Integer trailing timesteps tau_k = 999 - floor(1000 k / S), k < S."""
    return np.array([T_TRAIN - 1 - (T_TRAIN * k) // S for k in range(S)], dtype=np.int32)


def model_time(sampler: str, S: int) -> np.ndarray:
    """The time value fed to the timestep embedding at each step."""
    if sampler == "euler":
        return np.array([T_TRAIN * (1.0 - k / S) for k in range(S)], dtype=np.float64)
    return timesteps(S).astype(np.float64)


class Sampler:
    """One update rule; `step(k, x, out)` returns the next latent."""

    def __init__(self, kind: str, S: int, C: int):
        self.kind, self.S, self.C = kind, S, C
        self.ab = alpha_bar_table()
        self.tau = timesteps(S)
        self.prev_x0 = None
        self.prev_h = None

    def _a(self, k):
        return 1.0 if k >= self.S else float(self.ab[self.tau[k]])

    def step(self, k: int, x: np.ndarray, out: np.ndarray) -> np.ndarray:
        if self.kind == "ddim":
            eps = out[:, :self.C]
            a, a2 = self._a(k), self._a(k + 1)
            x0 = (x - math.sqrt(1.0 - a) * eps) / math.sqrt(a)
            return math.sqrt(a2) * x0 + math.sqrt(1.0 - a2) * eps
        if self.kind == "dpmpp2m":
            eps = out[:, :self.C]
            a = self._a(k)
            al, sg = math.sqrt(a), math.sqrt(1.0 - a)
            x0 = (x - sg * eps) / al
            if k == self.S - 1:
                return x0
            a2 = self._a(k + 1)
            al2, sg2 = math.sqrt(a2), math.sqrt(1.0 - a2)
            lam, lam2 = math.log(al / sg), math.log(al2 / sg2)
            h = lam2 - lam
            if k == 0:
                d = x0
            else:
                r = self.prev_h / h
                d = (1.0 + 1.0 / (2.0 * r)) * x0 - (1.0 / (2.0 * r)) * self.prev_x0
            self.prev_x0, self.prev_h = x0, h
            return (sg2 / sg) * x - al2 * (math.exp(-h) - 1.0) * d
        if self.kind == "euler":
            v = out[:, :self.C]
            s, s2 = 1.0 - k / self.S, 1.0 - (k + 1) / self.S
            return x + (s2 - s) * v
        raise ValueError(self.kind)


def sample(model: Model, x_T: np.ndarray, mask: Sequence[int], K: int,
           labels=None, text=None, p: Optional[bary.Params] = None,
           trace: Optional[Dict[str, list]] = None, cfg_scale: Optional[float] = None) -> np.ndarray:
    """The BaryCache sampling loop (Sec. 3.3) from x_T; returns the final latent.

    `cfg_scale` (class-conditional DiT only): classifier-free guidance as the
    paper's class-to-image runs use it (Sec. 4.1): the model runs on the batch
    twice, with the labels and with the null class (index n_classes), and the
    update takes out_u + s (out_c - out_u).  The stepwise feature, and so the
    cache, covers both halves.

    `trace`, if given, collects per step: 'feat' (the stepwise feature used),
    'out' (model output, guided) and 'x' (latent after the update)."""
    cfg = model.cfg
    S = len(mask)
    B = x_T.shape[0]
    steps = bary.plan(mask, K, None, p)
    ring = bary.Ring(K)
    tin = model_time(cfg.sampler, S)
    smp = Sampler(cfg.sampler, S, cfg.in_ch)
    ctx = model.context(text) if cfg.kind != "dit" else None
    guided = cfg_scale is not None
    if guided:
        if cfg.kind != "dit" or not cfg.n_classes:
            raise ValueError("classifier-free guidance needs a class-conditional DiT")
        labels = np.concatenate([np.asarray(labels), np.full(B, cfg.n_classes, dtype=np.int64)])
    Bm = 2 * B if guided else B
    x = np.asarray(x_T, dtype=np.float64)
    for k in range(S):
        cond = model.condition(tin[k], Bm, labels, text)
        if mask[k]:
            feat = model.stack(model.embed(np.concatenate([x, x]) if guided else x), cond, ctx)
            ring.push(feat, k)
        else:
            st = steps[k]
            feat = bary.forecast([ring.slots[i] for i in st.slots], st.w)
        out = np.asarray(model.final(feat, cond), dtype=np.float64)
        if guided:
            out = out[B:] + cfg_scale * (out[:B] - out[B:])
        x = smp.step(k, x, out)
        if trace is not None:
            trace.setdefault("feat", []).append(feat)
            trace.setdefault("out", []).append(out)
            trace.setdefault("x", []).append(x)
    return x
