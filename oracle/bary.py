"""Oracle: the Barycentric Extrapolator and the BaryCache cache context.

TEST INFRASTRUCTURE ONLY.  This is a plain, slow, fp64 CPU statement of what
the GPU path computes; only the tests, the smoke check and the benchmark's CPU
baseline may import it.  It shares no code with the HIP library.

Paper: "Memory-Efficient Training-Free Acceleration of Diffusion Transformers
with BaryCache", Sec. 3.2 (Barycentric Extrapolator, Eqs. 6-12) and Sec. 3.3
(BaryCache, Eq. 13).

Readings of the paper taken here (each also listed in the design notes):
  * nodes are ordered newest first: s_1 is the time of the most recent cached
    feature x_{f=-1} (Sec. 3.2, "Get Key" and "Get Raw Weight");
  * the blend of Eq. 12 mixes the barycentric estimate with the most recent
    feature: w = (1-lambda)*alpha + lambda*e_1 (the prose of Sec. 3.2 around
    Eq. 12 and the lambda ablation, Table 6).  The printed formula, which puts
    lambda on the oldest node, is kept as an option ("literal");
  * delta_H for H > 4, which the paper does not give, is 0.7 (the H = 4 value);
    delta_1 = 1;
  * the node coordinate of sampling step k is k itself, so |t - s_j| >= 1 and
    the clip of Eq. 10 is inactive inside the sampler;
  * a clipped sum that cancels to zero is an error (DEGENERATE);
  * while fewer than H features are cached, the available ones are used with
    delta of that count;
  * the full/forecast cadence "N": step k is full iff k mod N == 0 or k is the
    last step.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

# Constants the paper fixes (Sec. 3.2): clip bound C (Eq. 10), eta (after
# Eq. 12) and the decay table delta_H (before Eq. 11; also the history-length
# ablation).
CLIP_C = 10.0
ETA = 1e-12
DELTA_TABLE = {1: 1.0, 2: 1.0, 3: 0.95, 4: 0.7}
MAX_K = 8


class Degenerate(ValueError):
    """The normaliser of Eq. 11 vanished or is not finite."""


def delta_for(K: int) -> float:
    """delta_H of Sec. 3.2 (0.7 beyond the published H = 4 entry)."""
    return DELTA_TABLE.get(K, 0.7)


@dataclass
class Params:
    nodes: str = "trapezoid"   # "trapezoid" (Eq. 8-9) or "lagrange" (classical weights)
    C: float = CLIP_C          # clip bound of Eq. 10; math.inf disables the clip
    eta: float = ETA           # the small constant inside Eq. 11
    delta: Optional[float] = None  # None: delta_H from the table for H = K
    lam: float = 0.0           # blend factor of Eq. 12
    blend: str = "recent"      # "recent" (reading above) or "literal" (Eq. 12 as printed)


def trapezoid_coeffs(K: int) -> List[float]:
    """Eq. 8: c_1 = c_H = 1/2, interior c_j = 1 (K = 1: c_1 = 1/2)."""
    if K == 1:
        return [0.5]
    return [0.5] + [1.0] * (K - 2) + [0.5]


def node_weights(s: Sequence[float], mode: str) -> List[float]:
    """Numerators b_j of u_j = b_j / (t - s_j).

    trapezoid: b_j = (-1)^j c_j with j counted from 1 (Eq. 9).
    lagrange: the classical barycentric weights b_j = 1 / prod_{m != j}(s_j - s_m)."""
    K = len(s)
    if mode == "trapezoid":
        c = trapezoid_coeffs(K)
        return [c[j] * (-1.0) ** (j + 1) for j in range(K)]
    if mode == "lagrange":
        out = []
        for j in range(K):
            p = 1.0
            for m in range(K):
                if m != j:
                    p *= (s[j] - s[m])
            out.append(1.0 / p)
        return out
    raise ValueError(f"unknown node mode {mode!r}")


def validate_nodes(s: Sequence[float], t: float, mode: str) -> None:
    K = len(s)
    if not (1 <= K <= MAX_K):
        raise ValueError(f"K={K} outside [1, {MAX_K}]")
    if not all(math.isfinite(v) for v in list(s) + [t]):
        raise ValueError("non-finite node or query")
    if mode == "trapezoid" and K > 1:
        inc = all(s[j] < s[j + 1] for j in range(K - 1))
        dec = all(s[j] > s[j + 1] for j in range(K - 1))
        if not (inc or dec):
            raise ValueError("trapezoid nodes must be strictly monotone")
    if mode == "lagrange" and len(set(s)) != K:
        raise ValueError("lagrange nodes must be distinct")


def raw_weights(s: Sequence[float], t: float, mode: str) -> List[float]:
    """Eq. 9: u_j = b_j / (t - s_j).  A query exactly on a node gives
    +-inf in trapezoid mode (clipped later by Eq. 10)."""
    b = node_weights(s, mode)
    u = []
    for bj, sj in zip(b, s):
        d = t - sj
        u.append(bj / d if d != 0.0 else math.copysign(math.inf, bj))
    return u


def bary_weights(s: Sequence[float], t: float, p: Optional[Params] = None) -> np.ndarray:
    """The weight vector W of Eq. 12 for nodes s (newest first) and query t.

    Steps: raw weights (Eq. 9), clip (Eq. 10), signed power with eta and
    normalisation (Eq. 11), blend (Eq. 12)."""
    p = p or Params()
    s = [float(v) for v in s]
    t = float(t)
    validate_nodes(s, t, p.nodes)
    K = len(s)
    if p.nodes == "lagrange" and t in s:
        # The classical interpolant returns the node value itself.
        alpha = [1.0 if sj == t else 0.0 for sj in s]
    else:
        u = raw_weights(s, t, p.nodes)
        ut = [max(-p.C, min(p.C, uj)) for uj in u]                      # Eq. 10
        d = delta_for(K) if p.delta is None else p.delta
        v = [math.copysign(1.0, x) * (abs(x) + p.eta) ** d if x != 0.0 else 0.0
             for x in ut]                                                # Eq. 11 numerator
        total = sum(v)
        vmax = max(abs(x) for x in v)
        if not math.isfinite(total) or abs(total) <= 1e-12 * vmax or vmax == 0.0:
            raise Degenerate(f"normaliser {total!r} for nodes {s} and query {t}")
        alpha = [x / total for x in v]
    lam = p.lam
    if p.blend == "recent":
        w = [(1.0 - lam) * a for a in alpha]
        w[0] += lam
    elif p.blend == "literal":
        w = [(1.0 - lam) * a for a in alpha[:-1]] + [lam * alpha[-1]]
    else:
        raise ValueError(f"unknown blend {p.blend!r}")
    return np.array(w, dtype=np.float64)


# ---------------------------------------------------------------------------
# Full/forecast mask, cache context and the per-step plan (Sec. 3.3)
# ---------------------------------------------------------------------------

def make_mask(S: int, interval: int, force_last: bool = True) -> np.ndarray:
    """uint8 [S]: 1 = full step.  Step k is full iff k mod N == 0, or it is the
    last step (when force_last)."""
    if S < 1 or interval < 1:
        raise ValueError("S and interval must be >= 1")
    m = np.zeros(S, dtype=np.uint8)
    for k in range(S):
        if k % interval == 0 or (force_last and k == S - 1):
            m[k] = 1
    return m


class Ring:
    """The cache context H_t of Eq. 6 as K slots plus a head index.

    A full step stores its feature in slot (head+1) mod K, which evicts the
    oldest entry once K features are held; node j = 1..count (newest first)
    lives in slot (head - j + 1) mod K."""

    def __init__(self, K: int):
        if not (1 <= K <= MAX_K):
            raise ValueError("K out of range")
        self.K = K
        self.head = -1
        self.count = 0
        self.slots: List[Optional[np.ndarray]] = [None] * K
        self.coord: List[Optional[float]] = [None] * K

    def push(self, feat: Optional[np.ndarray], coord: float) -> int:
        self.head = (self.head + 1) % self.K
        self.slots[self.head] = feat
        self.coord[self.head] = float(coord)
        self.count = min(self.count + 1, self.K)
        return self.head

    def node_slots(self) -> List[int]:
        return [(self.head - j) % self.K for j in range(self.count)]

    def nodes(self) -> List[float]:
        return [self.coord[i] for i in self.node_slots()]


@dataclass
class PlanStep:
    is_full: bool
    count: int            # nodes used by a forecast step; nodes held after a full step
    head: int             # head after the step
    slots: List[int] = field(default_factory=list)   # forecast: slot of node j (newest first)
    w: List[float] = field(default_factory=list)     # forecast: weights, same order


def plan(mask: Sequence[int], K: int, coords: Optional[Sequence[float]] = None,
         p: Optional[Params] = None) -> List[PlanStep]:
    """Everything the sampling loop needs that does not depend on features:
    for each step, full or forecast; ring slot bookkeeping; forecast weights.
    The weights depend only on the schedule, which is what lets them be
    computed before the loop (Sec. 1, "online decoupling"; Sec. 3.2, Get Key)."""
    S = len(mask)
    coords = list(range(S)) if coords is None else [float(c) for c in coords]
    if S < 1 or int(mask[0]) != 1:
        raise ValueError("the first step must be a full step")
    p = p or Params()
    ring = Ring(K)
    out: List[PlanStep] = []
    for k in range(S):
        if mask[k]:
            ring.push(None, coords[k])
            out.append(PlanStep(True, ring.count, ring.head))
        else:
            s = ring.nodes()
            w = bary_weights(s, coords[k], p)   # delta of the node count in use
            out.append(PlanStep(False, ring.count, ring.head, ring.node_slots(), list(w)))
    return out


def forecast(feats: Sequence[np.ndarray], w: Sequence[float]) -> np.ndarray:
    """Eq. 13: x_hat = W H^T, the weighted sum of the cached features, in fp64."""
    acc = np.zeros(np.shape(feats[0]), dtype=np.float64)
    for wj, fj in zip(w, feats):
        acc += float(wj) * np.asarray(fj, dtype=np.float64)
    return acc
