"""Oracle of the runtime planner step (test infrastructure only).

Plain Python and numpy, written from Sec. 3.2 of the paper (the runtime
planner, Alg. 1) and its equations; only the test suite, the smoke check and
the benchmark's CPU-baseline leg may import it. It shares no code with the
library's planner (``csrc/pw_plan.cpp``) or its routing-statistics kernels.

Readings where the paper is silent (each also listed in the design notes):

* Planner units are page-table blocks (expert, projection, row block); the
  linear-block type u of a unit is gate_up for the gate and up projections and
  down for the down projection. Supported bitwidths are {16, 8, 4}; one
  planner step lowers a unit by one level (16 -> 8 or 8 -> 4), and a unit's
  8 -> 4 step becomes available only after its 16 -> 8 step was taken.
* Routing buckets: experts sorted by routing mass (descending, ties to the
  lower index); bucket j holds the experts from position floor(E * c_{j-1} + 1/2)
  up to floor(E * c_j + 1/2), c_j being the running sum of the fractions in
  float64 (the last bucket takes the rest).
* Bitwidth-floor stages: stage s gives every bucket a floor; a step b -> b' is
  legal at stage s when b' is not below the floor of the unit's bucket. Later
  stages relax the floors (the depth caps).
* Prompt residual heads are indexed by the linear-block type and the step
  (16 -> 8 or 8 -> 4); the features of a unit are its expert's features for
  the unit's type.
* Batched serving: request signals (routing masses and features) are averaged
  with the requests' KV-block weights; the residual head is linear in the
  features, so this averages the predicted residuals before clipping.
* GreedySelect: take the legal step with the smallest damage per released
  byte (ties: lower unit index, then the earlier step) until the bytes reach
  the target; if all legal steps do not reach it, the plan is all of them.
* SelectBestPlan: the strictest stage whose plan reaches the target (depth
  caps are relaxed only when the stricter ones cannot provide the bytes);
  if none does, the plan with the most bytes (ties: less damage, then the
  stricter stage).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

BITS = (16, 8, 4)
GATE_UP, DOWN_T = 0, 1


def target_bytes(free_blocks: int, threshold: int, kv_block_bytes: int) -> int:
    """Eq. 7: bytes to release for the KV cache under the current pressure."""
    return max(0, threshold + 1 - free_blocks) * kv_block_bytes


def global_damage(s_from: float, s_to: float) -> float:
    """Eq. 4: the offline sensitivity increase of lowering b -> b' (never negative)."""
    return max(s_to - s_from, 0.0)


def residual_scale(w: Sequence[float], a: float, c: float, phi: Sequence[float], alpha: float,
                   rho_min: float, rho_max: float) -> float:
    """Eqs. 5-6: the linear head's log residual, clipped, scaled and exponentiated."""
    rho = sum(float(wi) * float(pi) for wi, pi in zip(w, phi)) + float(a)
    rho = min(max(rho, rho_min), rho_max)
    return math.exp(alpha * c * rho)


def predicted_damage(mult: float, g: float, eta: float, eps: float) -> float:
    """Eq. 8: bucket multiplier times the prompt-adjusted damage, floored at eps."""
    return max(eps, mult * g * eta)


def routing_stats(rows: np.ndarray, row_of_slot: np.ndarray, topk_w: np.ndarray, offsets: np.ndarray,
                  sorted_slot: np.ndarray) -> np.ndarray:
    """Per expert, over its routed slots (Eq. 1's numerator and the routed-input
    features of Sec. 3.2): [sum r, count, sum r |x|, sum r |x|^2, max |x|],
    where r is the slot's routing weight and |x| the Euclidean norm of the
    slot's input row, in float64 and in slot order."""
    E = len(offsets) - 1
    out = np.zeros((E, 5), np.float64)
    rw = np.asarray(topk_w, np.float64).reshape(-1)
    for e in range(E):
        for i in range(int(offsets[e]), int(offsets[e + 1])):
            s = int(sorted_slot[i])
            r = rw[s]
            x = np.asarray(rows[int(row_of_slot[i])], np.float64)
            n2 = float(np.sum(x * x))
            n = math.sqrt(n2)
            out[e, 0] += r
            out[e, 1] += 1.0
            out[e, 2] += r * n
            out[e, 3] += r * n2
            out[e, 4] = max(out[e, 4], n)
    return out


def mass_and_features(stats: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 1 mass per expert and the feature vector phi = (routing-weighted
    mean norm, routing-weighted RMS norm, max norm) from routing_stats."""
    tot = float(np.sum(stats[:, 0]))
    E = stats.shape[0]
    m = np.zeros(E)
    phi = np.zeros((E, 3))
    for e in range(E):
        r = stats[e, 0]
        m[e] = r / tot if tot > 0 else 0.0
        if r > 0:
            phi[e] = (stats[e, 2] / r, math.sqrt(stats[e, 3] / r), stats[e, 4])
    return m, phi


@dataclass
class Config:
    bucket_frac: List[float]
    mult: List[float]
    floors: List[List[int]]          # [stage][bucket]
    alpha: float = 1.0
    rho_min: float = -1.0
    rho_max: float = 1.0
    eps: float = 1e-9
    head_w: np.ndarray = field(default_factory=lambda: np.zeros((2, 2, 3)))   # [u][step][3]
    head_a: np.ndarray = field(default_factory=lambda: np.zeros((2, 2)))
    head_c: np.ndarray = field(default_factory=lambda: np.ones((2, 2)))


@dataclass
class Unit:
    expert: int
    utype: int                 # GATE_UP or DOWN_T
    nbytes: Tuple[int, int, int]   # M^16, M^8, M^4 (Eq. 3's sizes)
    sens: Tuple[float, float, float]   # s^16, s^8, s^4


def buckets(mass: np.ndarray, frac: Sequence[float]) -> np.ndarray:
    E = len(mass)
    order = sorted(range(E), key=lambda e: (-mass[e], e))
    b = np.zeros(E, np.int64)
    acc, start = 0.0, 0
    for j, f in enumerate(frac):
        acc += f
        end = E if j == len(frac) - 1 else int(math.floor(E * acc + 0.5))
        for pos in range(start, min(end, E)):
            b[order[pos]] = j
        start = max(start, end)
    return b


def _next(bits: int) -> int:
    return {16: 8, 8: 4}.get(bits, 0)


def _step_index(b: int) -> int:
    return 0 if b == 16 else 1


@dataclass
class Plan:
    stage: int
    steps: List[Tuple[int, int, int]]   # (unit, from, to), in the order taken
    nbytes: int
    damage: float

    def final(self) -> Dict[int, Tuple[int, int]]:
        """unit -> (committed bitwidth, bitwidth after all of the unit's steps)"""
        out: Dict[int, Tuple[int, int]] = {}
        for (i, b, bp) in self.steps:
            out[i] = (out[i][0] if i in out else b, bp)
        return out


def step_damage(cfg: Config, unit: Unit, bucket: int, phi: np.ndarray, b: int) -> float:
    bp = _next(b)
    g = global_damage(unit.sens[BITS.index(b)], unit.sens[BITS.index(bp)])
    t = _step_index(b)
    eta = residual_scale(cfg.head_w[unit.utype][t], cfg.head_a[unit.utype][t], cfg.head_c[unit.utype][t],
                         phi[unit.expert][unit.utype], cfg.alpha, cfg.rho_min, cfg.rho_max)
    return predicted_damage(cfg.mult[bucket], g, eta, cfg.eps)


def greedy_select(cfg: Config, units: Sequence[Unit], q: Sequence[int], bucket_of: np.ndarray,
                  phi: np.ndarray, stage: int, D: int) -> Plan:
    """ScoreActions + GreedySelect of one stage: cheapest damage per byte first."""
    cur = list(q)
    steps: List[Tuple[int, int, int]] = []
    total, dmg = 0, 0.0
    while total < D:
        best = None
        for i, u in enumerate(units):
            b = cur[i]
            bp = _next(b)
            if bp == 0 or bp < cfg.floors[stage][bucket_of[u.expert]]:
                continue
            delta = u.nbytes[BITS.index(b)] - u.nbytes[BITS.index(bp)]
            d = step_damage(cfg, u, bucket_of[u.expert], phi, b)
            key = (d / delta, i)
            if best is None or key < best[0]:
                best = (key, i, b, bp, delta, d)
        if best is None:
            break
        _, i, b, bp, delta, d = best
        steps.append((i, b, bp))
        cur[i] = bp
        total += delta
        dmg += d
    return Plan(stage, steps, total, dmg)


def plan_step(cfg: Config, units: Sequence[Unit], q: Sequence[int], mass: np.ndarray, phi: np.ndarray,
              free_blocks: int, threshold: int, kv_block_bytes: int) -> Tuple[int, List[Plan], Optional[Plan]]:
    """One step of Alg. 1: (D, the refreshed per-stage plans, the selected plan or None)."""
    D = target_bytes(free_blocks, threshold, kv_block_bytes)
    bucket_of = buckets(mass, cfg.bucket_frac)
    plans = [greedy_select(cfg, units, q, bucket_of, phi, s, D) for s in range(len(cfg.floors))]
    if D <= 0:
        return D, plans, None
    for p in plans:
        if p.nbytes >= D:
            return D, plans, p
    best = max(plans, key=lambda p: (p.nbytes, -p.damage, -p.stage))
    return D, plans, best


def merge_requests(masses: Sequence[np.ndarray], phis: Sequence[np.ndarray],
                   weights: Sequence[float]) -> Tuple[np.ndarray, np.ndarray]:
    """Batch-level table: request signals averaged with their KV-block weights."""
    W = float(sum(weights))
    m = sum(w * np.asarray(x, np.float64) for w, x in zip(weights, masses)) / W
    p = sum(w * np.asarray(x, np.float64) for w, x in zip(weights, phis)) / W
    return m, p
