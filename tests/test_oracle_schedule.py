"""Pins for the oracle's lifetimes (Sec. 4.1 Eq. schedule, Alg. 1) and its budget reading."""
import itertools
import math

import numpy as np
import pytest

from oracle import schedule as sch


def test_defaults():
    # S_min = ceil(T/10): the smallest integer >= 0.1 T
    for T in range(1, 130):
        s = sch.s_min_default(T)
        assert s >= 0.1 * T and s - 1 < 0.1 * T
    assert [sch.s_min_default(T) for T in (10, 64, 50, 100)] == [1, 7, 5, 10]
    assert sch.budget_layer_steps(35, 32, 64) == 716
    assert sch.budget_layer_steps(50, 4, 10) == 20
    assert sch.budget_layer_steps(70, 10, 50) == 350


def test_tau_mode_literal_cases():
    T, smin = 10, 1
    # Lambda/tau = j/T exactly -> S = j; just above -> j + 1; capped at T; floored at S_min
    assert list(sch.lifetimes_tau([0.3, 0.30000001, 1.0, 0.0, 5.0], T, 1.0, smin)) == [3, 4, 10, 1, 10]
    assert list(sch.lifetimes_tau([0.3], T, 0.5, smin)) == [6]
    assert list(sch.lifetimes_tau([0.01], T, 1.0, 3)) == [3]


def test_tau_mode_properties():
    rng = np.random.default_rng(0)
    for _ in range(50):
        L, T = rng.integers(1, 9), rng.integers(2, 30)
        smin = rng.integers(1, T + 1)
        lam = rng.random(L)
        tau = rng.uniform(0.05, 2.0)
        S = sch.lifetimes_tau(lam, T, tau, smin)
        assert np.all(S >= smin) and np.all(S <= T)
        order = np.argsort(lam)
        assert np.all(np.diff(S[order]) >= 0)  # monotone in the score


def _breakpoints(lam, T, smin):
    """All tau at which some unit's lifetime changes under Eq. schedule."""
    taus = set()
    for l, x in enumerate(lam):
        for j in range(1, T + 1):
            if x > 0:
                taus.add(T * x / j)
    return sorted(taus)


@pytest.mark.parametrize("seed", range(25))
def test_budget_matches_tau_sweep_bruteforce(seed):
    """For every total that Eq. schedule realises at some tau, the budget reading returns that
    exact schedule; totals in between are filled by the next increments in key order."""
    rng = np.random.default_rng(seed)
    L, T = int(rng.integers(1, 5)), int(rng.integers(2, 9))
    smin = int(rng.integers(1, max(2, T // 2) + 1))
    lam = rng.random(L)
    realised = {}
    bps = _breakpoints(lam, T, smin)
    probes = [bps[0] * 2, bps[-1] / 2] + [b * (1 + 1e-9) for b in bps] + [b * (1 - 1e-9) for b in bps]
    for tau in probes:
        S = sch.lifetimes_tau(lam, T, tau, smin)
        realised.setdefault(int(S.sum()), set()).add(tuple(S))
    for total, scheds in realised.items():
        assert len(scheds) == 1  # no ties in random scores: one schedule per total
        got = sch.lifetimes_budget(lam, T, total, smin)
        assert tuple(got.lifetimes) == next(iter(scheds))
        assert got.layer_steps == total
    # every feasible budget sums exactly and sits between its neighbouring tau schedules
    totals = sorted(realised)
    for n_star in range(L * smin, L * T + 1):
        got = sch.lifetimes_budget(lam, T, n_star, smin)
        assert got.layer_steps == n_star
        below = max(t for t in totals if t <= n_star)
        above = min(t for t in totals if t >= n_star)
        lo = np.array(next(iter(realised[below])))
        hi = np.array(next(iter(realised[above])))
        assert np.all(lo <= got.lifetimes) and np.all(got.lifetimes <= hi)


def test_budget_tie_breaks_to_lower_unit():
    T, smin = 8, 1
    lam = [0.5, 0.5, 0.5]
    got = sch.lifetimes_budget(lam, T, 3 + 1, smin)
    assert list(got.lifetimes) == [2, 1, 1]
    got = sch.lifetimes_budget(lam, T, 3 + 2, smin)
    assert list(got.lifetimes) == [2, 2, 1]
    assert got.cut_margin == 0.0
    # permuting equal scores never moves the extra step off unit 0
    got = sch.lifetimes_budget([0.2, 0.5, 0.5], T, 3 + 1, smin)
    assert list(got.lifetimes) == [1, 2, 1]


def test_budget_infeasible_and_zero_scores():
    with pytest.raises(ValueError):
        sch.lifetimes_budget([0.5, 0.4], 10, 1, 1)
    with pytest.raises(ValueError):
        sch.lifetimes_budget([0.5, 0.4], 10, 21, 1)
    got = sch.lifetimes_budget([0.0, 0.7], 10, 2 + 9, 1)
    assert list(got.lifetimes) == [1, 10]
    got = sch.lifetimes_budget([0.0, 0.7], 10, 2 + 10, 1)  # only then does the zero unit grow
    assert list(got.lifetimes) == [2, 10]


def test_budget_decreasing_order_freezes_low_scores_first():
    """Corollary 'Budgeted freezing': lower scores never outlive higher ones."""
    rng = np.random.default_rng(4)
    for _ in range(30):
        lam = rng.random(12)
        T = 20
        got = sch.lifetimes_budget(lam, T, int(rng.integers(12 * 2, 12 * 20)), 2)
        order = np.argsort(lam)
        assert np.all(np.diff(got.lifetimes[order]) >= 0)


def test_active_mask():
    S = [3, 1, 5]
    m = sch.active_mask(S, 5)
    assert m.shape == (5, 3)
    assert list(m.sum(axis=0)) == S
    assert np.all(m[0] == 1)
    # nested in s: once frozen, frozen for good
    assert np.all(np.diff(m.astype(int), axis=0) <= 0)
