"""Oracle replay (oracle): the non-deployable headroom search of the input-aware baselines.

Test infrastructure: only the tests, the smoke check and the benchmark's CPU baseline use
this module; the product path never imports it.

Appendix "Protocol Details", paragraph "Oracle replay" (Tables "LLaDA-8B language
evaluation" and "Static versus input-aware scheduling at matched per-step active counts"):
the search first records the full (unscheduled) trajectory; at step s it greedily grows a
cumulative frozen set F_s: every remaining unit j is tried frozen together with F_s, the
output deviation
    delta(F_s + {j}, s) = ||eps^(F_s + {j})(z_s, s) - eps(z_s, s)||_2 / (||eps(z_s, s)||_2 + 1e-8)
is measured, and the candidate of least deviation (ties to the lower unit index) is added
while the deviation stays at most tau_agree (5e-3 in the paper).  A global ceiling bounds
the active layer-steps of the trajectory.

Readings where the paper is silent:
* z_s is the recorded unscheduled trajectory's state, and a frozen unit adds the update it
  produced in the unscheduled evaluation of its last active step (the search needs no
  other trajectory);
* step 1 is full (no cached update exists yet), and F_s starts from F_{s-1}: once frozen, a
  unit stays frozen, so the result is a nested schedule with S_l = the step before unit l
  joined F;
* the deviation is measured on the rows the sampler updates (LLaDA: the masked response
  positions; U-ViT: the patch tokens; all rows otherwise), over the whole batch;
* the ceiling: while keeping the current active count for the remaining steps would exceed
  it, candidates keep joining F in the same least-deviation order, regardless of the
  tolerance.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from . import model as om

DEV_EPS = 1e-8


def deviation(eps: np.ndarray, ref: np.ndarray, rows) -> float:
    """||eps - ref||_2 / (||ref||_2 + 1e-8) over rows [r0, r1) of every sample."""
    r0, r1 = rows
    e = np.asarray(eps, np.float64)[:, r0:r1]
    r = np.asarray(ref, np.float64)[:, r0:r1]
    return float(np.sqrt(np.sum((e - r) ** 2)) / (np.sqrt(np.sum(r * r)) + DEV_EPS))


@dataclass
class ReplayResult:
    lifetimes: np.ndarray
    order: List[tuple] = field(default_factory=list)        # (step, unit) in the order units joined F
    log: Dict[tuple, float] = field(default_factory=dict)   # (step, round, unit) -> deviation
    evaluations: int = 0


def search(model: om.Model, z0: np.ndarray, tau_agree: float = 5e-3,
           max_layer_steps: Optional[int] = None) -> ReplayResult:
    cfg = model.cfg
    L, T = model.n_units, cfg.T  # scheduled units: blocks or branches
    ceiling = max_layer_steps if max_layer_steps and max_layer_steps > 0 else L * T
    cross = [model.cross_kv(u) for u in model.units] if model.arch in om.CROSS_ARCHS else None
    z = np.array(z0, dtype=np.float64)
    frozen = [False] * L
    S = np.full(L, T, dtype=np.int64)
    last_update: Dict[int, np.ndarray] = {}  # unit -> update of its latest active step
    out = ReplayResult(S)
    spent = 0
    for s in range(1, T + 1):
        updates: Dict[int, np.ndarray] = {}
        ref = om.denoise_step(model, z, s, [1] * L, updates, cross)  # unscheduled; records every update
        out.evaluations += 1
        nfrozen = sum(frozen)
        rnd = 0
        while s > 1 and nfrozen < L:
            cand = [l for l in range(L) if not frozen[l]]
            devs = {}
            for j in cand:
                row = [0 if (frozen[l] or l == j) else 1 for l in range(L)]
                eps = om.denoise_step(model, z, s, row, dict(last_update), cross)
                out.evaluations += 1
                devs[j] = deviation(eps, ref, cfg.update_rows)
                out.log[(s, rnd, j)] = devs[j]
            best = min(cand, key=lambda j: (devs[j], j))
            planned = spent + (T - s + 1) * (L - nfrozen)
            if devs[best] > tau_agree and planned <= ceiling:
                break
            frozen[best] = True
            S[best] = s - 1
            out.order.append((s, best))
            nfrozen += 1
            rnd += 1
        spent += L - nfrozen
        for l in range(L):
            if not frozen[l]:
                last_update[l] = updates[l]
        z = om.sampler_update(cfg, z, ref, s)
    out.lifetimes = S
    return out
