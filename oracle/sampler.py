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
  * Euler on the flow-matching ODE with sigma_k = 1 - k/S, model time 1000 sigma;
    optionally time-shifted, sigma -> s sigma / (1 + (s - 1) sigma), the
    schedule the published video model samples with (shift 7).
The loop itself is Sec. 3.3: on a full step run the stack and store its output
in the cache; otherwise forecast it from the cache with Eq. 13; then the final
layer and the sampler update.

The adaptive schedule (Sec. 4.5, Table 5) is described only as a TeaCache-style
rule: relative changes of a feature probe accumulate, and a full step runs when
the accumulated drift reaches the threshold l.  Readings taken here: the probe
is the first block's modulated attention input (Model.probe) at the current
latent and step; the change at step k is the relative L1 distance
sum|p_k - p_{k-1}| / sum|p_{k-1}| over the whole batch (no rescaling
polynomial: its coefficients are fitted to trained weights); steps 0 and S-1
always run the stack; a full step resets the accumulator to zero.

Blockwise mode (Sec. 4.5, Tables 5 and 6) caches every module's output instead
of the stack's.  The paper fixes only its two ends (Br = 1 is stepwise
caching; the blockwise rows of Table 5 take Br = 0); what is built is Br = 0:
a full step keeps each module's output before its gate (attention, PixArt's
cross-attention, MLP) in a ring of its own, and a skipped step embeds the
current latent and adds, block by block, each module's forecast (Eq. 13 with
the same weights for every site) times the current step's gate.
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


def shifted_sigma(sigma, shift: float = 1.0):
    """The time shift of a flow-matching schedule: s sigma / (1 + (s - 1) sigma)
    (s = 1: unchanged).  It keeps 0 and 1 fixed and, for s > 1, spends more of
    the steps at high noise."""
    return shift * sigma / (1.0 + (shift - 1.0) * sigma)


def flow_sigma(k: int, S: int, shift: float = 1.0) -> float:
    return shifted_sigma(1.0 - k / S, shift)


def model_time(sampler: str, S: int, shift: float = 1.0) -> np.ndarray:
    """The time value fed to the timestep embedding at each step."""
    if sampler == "euler":
        return np.array([T_TRAIN * flow_sigma(k, S, shift) for k in range(S)], dtype=np.float64)
    return timesteps(S).astype(np.float64)


class Sampler:
    """One update rule; `step(k, x, out)` returns the next latent."""

    def __init__(self, kind: str, S: int, C: int, shift: float = 1.0):
        self.kind, self.S, self.C, self.shift = kind, S, C, shift
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
            s, s2 = flow_sigma(k, self.S, self.shift), flow_sigma(k + 1, self.S, self.shift)
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
    shift = getattr(cfg, "flow_shift", 1.0)
    tin = model_time(cfg.sampler, S, shift)
    smp = Sampler(cfg.sampler, S, cfg.in_ch, shift)
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


def relative_l1(cur: np.ndarray, prev: np.ndarray) -> float:
    """sum|cur - prev| / sum|prev| over every element (0/0 = 0, x/0 = inf)."""
    num = float(np.abs(np.asarray(cur, np.float64) - np.asarray(prev, np.float64)).sum())
    den = float(np.abs(np.asarray(prev, np.float64)).sum())
    if den == 0.0:
        return 0.0 if num == 0.0 else math.inf
    return num / den


class AdaptiveRule:
    """The accumulate-and-trigger decision of the adaptive schedule: step k runs
    the stack if it is the first or the last step, or if the changes summed
    since the last full step reach `ell`; a full step empties the sum."""

    def __init__(self, ell: float, S: int):
        if not ell >= 0.0:
            raise ValueError("the threshold must be >= 0")
        self.ell, self.S, self.acc = float(ell), S, 0.0
        self.compared = 0.0   # the sum the last decision compared with ell

    def full(self, k: int, change: float) -> bool:
        if k == 0 or k == self.S - 1:
            self.acc = self.compared = 0.0
            return True
        self.acc += change
        self.compared = self.acc
        if self.acc >= self.ell:
            self.acc = 0.0
            return True
        return False


def adaptive_mask(changes: Sequence[float], ell: float) -> List[int]:
    """The mask the rule gives for a fixed sequence of changes (changes[0] is
    unused: step 0 has no previous probe)."""
    rule = AdaptiveRule(ell, len(changes))
    return [1 if rule.full(k, float(c)) else 0 for k, c in enumerate(changes)]


def sample_adaptive(model: Model, x_T: np.ndarray, S: int, ell: float, K: int, labels=None, text=None,
                    p: Optional[bary.Params] = None, trace: Optional[Dict[str, list]] = None):
    """The sampling loop under the adaptive schedule: at every step the probe
    decides (AdaptiveRule) whether the stack runs; a skipped step forecasts
    with the weights of the full steps taken so far (Eq. 8-13: the plan of a
    step depends only on the steps before it).

    Returns (final latent, realised mask, changes); changes[k] is the probe's
    relative L1 change at step k >= 1 (changes[0] = 0)."""
    cfg = model.cfg
    B = x_T.shape[0]
    ring = bary.Ring(K)
    shift = getattr(cfg, "flow_shift", 1.0)
    tin = model_time(cfg.sampler, S, shift)
    smp = Sampler(cfg.sampler, S, cfg.in_ch, shift)
    ctx = model.context(text) if cfg.kind != "dit" else None
    rule = AdaptiveRule(ell, S)
    x = np.asarray(x_T, dtype=np.float64)
    mask: List[int] = []
    changes: List[float] = []
    prev = None
    for k in range(S):
        cond = model.condition(tin[k], B, labels, text)
        emb = model.embed(x)
        pr = model.probe(emb, cond)
        change = relative_l1(pr, prev) if k > 0 else 0.0
        prev = pr
        full = rule.full(k, change)
        if trace is not None:
            trace.setdefault("acc", []).append(rule.compared)
        mask.append(1 if full else 0)
        changes.append(change)
        if full:
            feat = model.stack(emb, cond, ctx)
            ring.push(feat, k)
        else:
            st = bary.plan(mask, K, None, p)[k]
            feat = bary.forecast([ring.slots[i] for i in st.slots], st.w)
        out = np.asarray(model.final(feat, cond), dtype=np.float64)
        x = smp.step(k, x, out)
        if trace is not None:
            trace.setdefault("feat", []).append(feat)
            trace.setdefault("probe", []).append(pr)
            trace.setdefault("x", []).append(x)
    return x, mask, changes


def sample_blockwise(model: Model, x_T: np.ndarray, mask: Sequence[int], K: int, labels=None, text=None,
                     p: Optional[bary.Params] = None, trace: Optional[Dict[str, list]] = None) -> np.ndarray:
    """The sampling loop in blockwise mode (Br = 0) for DiT and PixArt models:
    the cache holds every module site of every block (one ring slot is the list
    of the sites' outputs of one full step)."""
    cfg = model.cfg
    if cfg.kind not in ("dit", "pixart"):
        raise ValueError("blockwise mode is built for DiT and PixArt blocks")
    S = len(mask)
    B = x_T.shape[0]
    steps = bary.plan(mask, K, None, p)
    ring = bary.Ring(K)
    shift = getattr(cfg, "flow_shift", 1.0)
    tin = model_time(cfg.sampler, S, shift)
    smp = Sampler(cfg.sampler, S, cfg.in_ch, shift)
    ctx = model.context(text) if cfg.kind != "dit" else None
    x = np.asarray(x_T, dtype=np.float64)
    for k in range(S):
        cond = model.condition(tin[k], B, labels, text)
        emb = model.embed(x)
        h = emb
        if mask[k]:
            sites: list = []
            for l in range(cfg.depth):
                h = model.dit_block(l, h, model.block_mod(l, cond), ctx, modules=sites)
            ring.push(sites, k)
        else:
            st = steps[k]
            nodes = [ring.slots[i] for i in st.slots]
            i = 0
            for l in range(cfg.depth):
                for g in model.module_gates(l, model.block_mod(l, cond)):
                    h = h + g[:, None, :] * bary.forecast([n[i] for n in nodes], st.w)
                    i += 1
        feat = h
        out = np.asarray(model.final(feat, cond), dtype=np.float64)
        if trace is not None:
            trace.setdefault("x_in", []).append(x)
            trace.setdefault("emb", []).append(emb)
            trace.setdefault("feat", []).append(feat)
        x = smp.step(k, x, out)
    return x
