"""Pins for the causal activation-drift policy of the oracle (appendix "Protocol Details",
"Dynamic baselines"; Table "Static versus input-aware scheduling at matched per-step active
counts")."""
import functools

import numpy as np
import pytest

import synth
from oracle import drift as od
from oracle import model as om
from oracle import schedule as osch
from oracle import spectral as osp


@functools.lru_cache(maxsize=None)
def load(name, **kw):
    cfg = synth.get_config(name, **kw)
    return cfg, synth.model_weights(cfg), synth.inputs(cfg)


def static_mask(cfg, w, pct):
    raw = [osp.unit_score(osp.unit_matrices(u, cfg.d, cfg.dtype), cfg.dh).raw for u in w]
    n = osch.budget_layer_steps(pct, cfg.L, cfg.T)
    S = osch.lifetimes_budget(osp.normalise(raw), cfg.T, n, osch.s_min_default(cfg.T)).lifetimes
    return osch.active_mask(S, cfg.T)


def test_select_top_m_ties_to_lower_index():
    assert od.select([0.5, 0.9, 0.9, 0.1], 2).tolist() == [0, 1, 1, 0]
    assert od.select([0.5, 0.9, 0.9, 0.1], 1).tolist() == [0, 1, 0, 0]
    assert od.select([0.3, 0.3, 0.3, 0.3], 2).tolist() == [1, 1, 0, 0]
    assert od.select([0.0, 1.0, 0.0, 1.0], 3).tolist() == [1, 1, 0, 1]
    assert od.select([1.0, 2.0], 0).tolist() == [0, 0]
    assert od.select([1.0, 2.0], 2).tolist() == [1, 1]


def test_drift_formula():
    a = np.array([[3.0, 4.0]])
    assert od.drift(a, a) == 0.0
    assert od.drift(a, np.zeros_like(a)) == pytest.approx(5.0 / (5.0 + 1e-8), rel=1e-15)
    assert od.drift(np.zeros((2, 2)), np.ones((2, 2))) == pytest.approx(2.0 / 1e-8)


@pytest.mark.parametrize("name", ["tiny_ragged", "llada_mini"])
def test_policy_counts_first_step_and_unit0_drift(name):
    """First step full; m_s active units at every step; the drift of unit 0 is the drift of
    the step's initial stream h_0 = z_s, computed here from the trajectory's own states."""
    cfg, w, x = load(name)
    m = om.Model(cfg, w, x)
    mask = static_mask(cfg, w, cfg.budgets[-1])
    tr = od.trajectory(m, x["z"], mask)
    assert tr.active[0].tolist() == [1] * cfg.L
    for s in range(1, cfg.T + 1):
        assert int(tr.active[s - 1].sum()) == int(mask[s - 1].sum())
        assert np.array_equal(tr.active[s - 1], od.select(tr.drift[s - 1], int(mask[s - 1].sum())) if s > 1
                              else np.ones(cfg.L, np.uint8))
    zs = [np.asarray(x["z"], np.float64)] + tr.z  # z_1, z_2, ...
    for s in range(3, cfg.T + 1):
        a, b = zs[s - 2], zs[s - 3]  # z_{s-1}, z_{s-2}
        want = np.sqrt(np.sum((a - b) ** 2)) / (np.sqrt(np.sum(a * a)) + 1e-8)
        assert tr.drift[s - 1][0] == pytest.approx(want, rel=1e-12)
    assert np.all(tr.drift[1] == 0.0)  # no lagged drift at step 2
    assert any(not np.array_equal(tr.active[s], mask[s]) for s in range(cfg.T))  # input-dependent sets


def test_all_active_budget_is_the_unscheduled_trajectory():
    cfg, w, x = load("llada_mini")
    m = om.Model(cfg, w, x)
    ones = np.ones((cfg.T, cfg.L), np.uint8)
    tr = od.trajectory(m, x["z"], ones, steps=4)
    ref = om.trajectory(m, x["z"], None, steps=4)
    for a, b in zip(tr.z, ref.z):
        assert np.array_equal(a, b)


def test_reactivated_unit_refreshes_its_cache():
    """A unit frozen, then active, then frozen again adds the update of its latest active
    step: the second frozen step equals a run where that update is injected by hand."""
    cfg, w, x = load("tiny_ragged")
    m = om.Model(cfg, w, x)
    rows = np.ones((cfg.T, cfg.L), np.uint8)
    rows[1, 1] = 0   # step 2: unit 1 frozen (update of step 1)
    rows[3, 1] = 0   # step 4: unit 1 frozen (update of step 3)
    tr = od.trajectory(m, x["z"], rows, steps=4, forced_rows=rows)
    # replay by hand: record unit 1's update at step 3, then step 4 with it frozen
    cache = {}
    z = np.asarray(x["z"], np.float64)
    for s in range(1, 4):
        eps = om.denoise_step(m, z, s, rows[s - 1], cache)
        z = om.sampler_update(cfg, z, eps, s)
    d3 = cache[1].copy()
    h = om.initial_stream(m, z, 4)
    u0, _ = m.unit_active(0, h, om.timestep_value(4, cfg.T))
    h1 = u0 + d3
    h2, _ = m.unit_active(2, h1, om.timestep_value(4, cfg.T))
    z4 = om.sampler_update(cfg, z, h2, 4)
    assert np.array_equal(tr.z[3], z4)
    assert np.abs(d3).max() > 0
