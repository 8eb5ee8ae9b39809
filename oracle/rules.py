"""Static ranking rules for lifetimes at a matched layer-step budget (oracle).

Test infrastructure: only the tests, the smoke check and the benchmark's CPU baseline use
this package; the product path never imports it.

Sec. "Static ranking comparisons" and Table "Static rankings at matched layer-step budgets"
compare the SCR/Frobenius score with random, depth-only, Frobenius-norm, spectral-norm,
stable-rank, Frobenius x stable-rank and raw-SCR rankings, every one held to the same
layer-step budget, with larger raw scores receiving longer lifetimes.  The paper does not
spell the baselines out; the readings here are:

* A matrix rule keeps the unit's component structure (Eqs. app-attn-score,
  app-xattn-score, app-mlp-score, app-conv-score, app-block-score) and replaces the
  matrix score g(W) by the rule's statistic gamma(W):
    frob         ||W||_F
    spectral     ||W||_2
    stable_rank  ||W||_2^2 / ||W||_F^2   (the stable rank ||W||_F^2 / ||W||_2^2, oriented
                                          like SCR: a concentrated spectrum ranks high; the
                                          paper orients every baseline toward sensitivity
                                          and reports stable rank anti-correlated with SCR)
    frob_srank   ||W||_F * ||W||_2^2 / ||W||_F^2
    raw_scr      sqrt(rho(SCR_eta))        (g(W) without its Frobenius factor, so that the
                                          method is the Frobenius rule times the raw-SCR
                                          rule, matrix by matrix)
    scr_frob     g(W)                      (the method, Eq. app-matrix-score)
* depth: raw score l + 1 (0-based unit index l): deeper units live longer, the direction of
  the paper's own schedules (Table "Representative display lifetimes").
* random: the raw score of unit l is the (l+1)-th output of SplitMix64 seeded with the
  given seed, as a double in [0, 1): (x >> 11) * 2^-53.
* Every rule's raw scores go through Eq. app-score-normalization and the same budget
  reading as the method (``schedule.lifetimes_budget``).
"""
from __future__ import annotations

import math
from typing import Dict, Sequence

import numpy as np

from . import schedule as sch
from . import spectral as sp

RULES = ("scr_frob", "random", "depth", "frob", "spectral", "stable_rank", "frob_srank", "raw_scr")
MATRIX_RULES = ("scr_frob", "frob", "spectral", "stable_rank", "frob_srank", "raw_scr")

_MASK64 = (1 << 64) - 1


def splitmix64(seed: int, i: int) -> int:
    """Output i (i >= 1) of SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
    number generators", OOPSLA 2014): the state after i increments of the golden gamma
    0x9E3779B97F4A7C15, passed through Stafford's variant 13 of the MurmurHash3 64-bit finaliser."""
    z = (seed + i * 0x9E3779B97F4A7C15) & _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def random_raw(L: int, seed: int) -> np.ndarray:
    return np.array([(splitmix64(seed, l + 1) >> 11) * 2.0 ** -53 for l in range(L)], np.float64)


def depth_raw(L: int) -> np.ndarray:
    return np.arange(1, L + 1, dtype=np.float64)


def statistic(st: sp.MatrixStats, rule: str) -> float:
    """gamma(W) of a matrix rule from the matrix's statistics."""
    F = st.frob_sq
    if rule == "scr_frob":
        return st.g
    if rule == "frob":
        return math.sqrt(F)
    if rule == "spectral":
        return math.sqrt(st.sigma1_sq)
    if rule == "stable_rank":
        return st.sigma1_sq / F if F > 0 else 0.0
    if rule == "frob_srank":
        return math.sqrt(F) * (st.sigma1_sq / F) if F > 0 else 0.0
    if rule == "raw_scr":
        return st.g / math.sqrt(F) if F > 0 else 0.0
    raise ValueError(rule)


def unit_raw(stats: Dict[str, sp.MatrixStats], head_dim: int, rule: str) -> float:
    """The unit's raw score with gamma in place of g in the block equations."""
    g = {role: statistic(s, rule) for role, s in stats.items()}
    raw = 0.0
    if all(r in g for r in sp.ATTN_ROLES):
        raw += sp.q_attn(g["q"], g["k"], g["v"], g["o"], head_dim)
    if all(r in g for r in sp.XATTN_ROLES):
        raw += sp.q_attn(g["xq"], g["xk"], g["xv"], g["xo"], head_dim)
    if all(r in g for r in sp.MLP_ROLES):
        raw += sp.q_mlp(g["w1"], g["w2"])
    for role in sorted(g):
        if role.startswith("conv"):
            raw += sp.q_conv(g[role])
    return raw


def raw_scores(rule: str, unit_stats: Sequence[Dict[str, sp.MatrixStats]], head_dim: int, seed: int = 0,
               L: int = 0) -> np.ndarray:
    """Raw scores of every unit under ``rule`` (``unit_stats`` may be empty for the unit rules)."""
    L = L or len(unit_stats)
    if rule == "random":
        return random_raw(L, seed)
    if rule == "depth":
        return depth_raw(L)
    return np.array([unit_raw(s, head_dim, rule) for s in unit_stats], np.float64)


def lifetimes(rule: str, unit_stats, head_dim: int, T: int, n_star: int, s_min: int, seed: int = 0,
              L: int = 0) -> sch.BudgetSchedule:
    """Lifetimes of ``rule`` at exactly ``n_star`` layer-steps (the method's budget reading)."""
    raw = raw_scores(rule, unit_stats, head_dim, seed, L)
    return sch.lifetimes_budget(sp.normalise(raw), T, n_star, s_min)
