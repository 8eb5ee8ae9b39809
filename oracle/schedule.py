"""Static lifetimes from normalised unit scores (oracle).

Sec. 4.1, Eq. schedule:  S_l = max{S_min, ceil(T min(1, Lambda_hat_l / tau))}
and Alg. 1 (score every matrix, combine, normalise, apply Eq. schedule).

Readings where the paper is silent:
* S_min defaults to ceil(T / 10), the smallest integer >= 0.1 T.
* A percentage budget is the integer ceiling N* = floor(pct L T / 100)
  layer-steps.
* Budget mode sweeps Eq. schedule over tau.  As 1/tau grows, unit l gains
  its (j+1)-th step exactly when T Lambda_hat_l / tau > j, i.e. at key
  kappa = j / Lambda_hat_l.  Granting these events in increasing kappa
  order reproduces Eq. schedule at every tau; the budget is then filled to
  exactly N* by the next events, ties broken by the lower unit index and
  then the lower j (the paper breaks ties toward the lower unit index in
  its dynamic baselines).  Corollary "Budgeted freezing" motivates the
  order: freeze in increasing Lambda_hat.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np


def s_min_default(T: int) -> int:
    """ceil(T / 10) in integers."""
    return (T + 9) // 10


def budget_layer_steps(pct: int, L: int, T: int) -> int:
    """floor(pct * L * T / 100) in integers."""
    return (pct * L * T) // 100


def lifetimes_tau(scores: Sequence[float], T: int, tau: float, s_min: int) -> np.ndarray:
    """Eq. schedule, evaluated literally in float64."""
    out = []
    for lam in scores:
        out.append(max(s_min, int(math.ceil(T * min(1.0, lam / tau)))))
    return np.asarray(out, dtype=np.int64)


@dataclass
class BudgetSchedule:
    lifetimes: np.ndarray   # S_l
    layer_steps: int        # sum_l S_l (== N*)
    cut_margin: float       # relative gap between the first refused and last granted key


def lifetimes_budget(scores: Sequence[float], T: int, n_star: int, s_min: int) -> BudgetSchedule:
    """Eq. schedule swept over tau until exactly N* layer-steps are granted."""
    lam = np.asarray(scores, dtype=np.float64)
    L = lam.size
    if n_star < L * s_min or n_star > L * T:
        raise ValueError("infeasible budget")
    events = []
    for l in range(L):
        for j in range(s_min, T):
            key = (j / lam[l]) if lam[l] > 0 else math.inf
            events.append((key, l, j))
    events.sort()
    grant = n_star - L * s_min
    S = np.full(L, s_min, dtype=np.int64)
    for key, l, j in events[:grant]:
        S[l] += 1
    if 0 < grant < len(events):
        last, nxt = events[grant - 1][0], events[grant][0]
        margin = (nxt - last) / last if math.isfinite(last) and last > 0 else math.inf
        if not math.isfinite(nxt):
            margin = math.inf
    else:
        margin = math.inf
    return BudgetSchedule(S, int(S.sum()), margin)


def active_mask(lifetimes: Sequence[int], T: int) -> np.ndarray:
    """active[s-1, l] = (s <= S_l) for s = 1..T  (Alg. 2, the branch test)."""
    S = np.asarray(lifetimes, dtype=np.int64)
    s = np.arange(1, T + 1)[:, None]
    return (s <= S[None, :]).astype(np.uint8)
