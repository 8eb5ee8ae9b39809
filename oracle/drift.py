"""Causal activation-drift policy (oracle).

Test infrastructure: only the tests, the smoke check and the benchmark's CPU baseline use
this module; the product path never imports it.

Appendix "Protocol Details", paragraph "Causal activation drift" (the input-aware baseline
of Table "Static versus input-aware scheduling at matched per-step active counts"):

* after step s-1 the policy records, for every unit l, the lagged normalised drift
  d_{l,s-1} = ||h_{l-1,s-1} - h_{l-1,s-2}||_2 / (||h_{l-1,s-1}||_2 + 1e-8) of the unit's
  input h_{l-1} (the residual stream arriving at unit l);
* at step s it activates exactly m_s units, those with the largest d_{l,s-1}, where m_s is
  the static schedule's active count at step s; ties go to the lower unit index;
* the first step is full.

The active sets are therefore not nested in s: a unit may be frozen, then active again.
Alg. 2 refreshes a unit's cached update at every step on which it is active, so a frozen
unit adds the update of its most recent active step (``model.denoise_step`` does exactly
that for any active set).

Readings where the paper is silent:
* the norms are taken over the whole input tensor of the step (every sample, token and
  feature of the batch);
* the input of a U-ViT out-block is the stream before its skip linear;
* at step 2 there is no lagged drift (no step 0 exists), so every unit's drift counts as 0
  and the tie rule activates the m_2 lowest-indexed units.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from . import model as om

DRIFT_EPS = 1e-8


def drift(curr: np.ndarray, prev: np.ndarray) -> float:
    """||curr - prev||_2 / (||curr||_2 + 1e-8) over every element."""
    c = np.asarray(curr, np.float64)
    p = np.asarray(prev, np.float64)
    return float(np.sqrt(np.sum((c - p) ** 2)) / (np.sqrt(np.sum(c * c)) + DRIFT_EPS))


def select(drifts, m: int) -> np.ndarray:
    """The m units of largest drift, ties to the lower index, as a 0/1 row."""
    d = np.asarray(drifts, np.float64)
    order = sorted(range(d.size), key=lambda l: (-d[l], l))
    row = np.zeros(d.size, np.uint8)
    row[order[:m]] = 1
    return row


@dataclass
class DriftTrajectory:
    z: List[np.ndarray] = field(default_factory=list)       # z after each step
    active: List[np.ndarray] = field(default_factory=list)  # the row each step ran
    drift: List[np.ndarray] = field(default_factory=list)   # d_{l,s-1} each step's choice used


def trajectory(model: om.Model, z0: np.ndarray, static_mask: np.ndarray, steps: Optional[int] = None,
               forced_rows: Optional[np.ndarray] = None) -> DriftTrajectory:
    """Run the policy for steps 1..steps.  ``static_mask[s-1]`` supplies m_s.
    ``forced_rows`` (tests) replaces the policy's choice by given rows while still recording
    the drift the policy would have used."""
    cfg = model.cfg
    steps = cfg.T if steps is None else steps
    cross = [model.cross_kv(u) for u in model.units] if model.arch in om.CROSS_ARCHS else None
    cache: Dict[int, np.ndarray] = {}
    z = np.array(z0, dtype=np.float64)
    prev: Optional[Dict[int, np.ndarray]] = None
    prev2: Optional[Dict[int, np.ndarray]] = None
    out = DriftTrajectory()
    for s in range(1, steps + 1):
        m = int(np.asarray(static_mask[s - 1]).sum())
        U = model.n_units
        if prev is not None and prev2 is not None:
            d = np.array([drift(prev[l], prev2[l]) for l in range(U)])
        else:
            d = np.zeros(U)
        row = np.ones(U, np.uint8) if s == 1 else select(d, m)
        if forced_rows is not None:
            row = np.asarray(forced_rows[s - 1], np.uint8)
        inputs: Dict[int, np.ndarray] = {}
        eps = om.denoise_step(model, z, s, row, cache, cross, unit_inputs=inputs)
        z = om.sampler_update(cfg, z, eps, s)
        prev2, prev = prev, inputs
        out.z.append(z)
        out.active.append(row)
        out.drift.append(d)
    return out
