"""Pins for the oracle-replay search (appendix "Protocol Details", "Dynamic baselines",
"Oracle replay")."""
import functools

import numpy as np
import pytest

import synth
from oracle import model as om
from oracle import replay as orp


@functools.lru_cache(maxsize=None)
def load(name, **kw):
    cfg = synth.get_config(name, **kw)
    return cfg, synth.model_weights(cfg), synth.inputs(cfg)


def zero_units(w, units):
    """Weights where the listed units' branches output exactly zero (no biases in the tiny
    architecture): freezing such a unit changes nothing."""
    w = [dict(u) for u in w]
    for l in units:
        for key in ("w_o", "w2"):
            w[l][key] = np.zeros_like(w[l][key])
    return w


def test_deviation_formula():
    ref = np.zeros((2, 5, 3))
    ref[:, 1:4] = 2.0
    eps = ref.copy()
    eps[0, 2, 0] += 3.0
    eps[1, 0, 0] += 100.0  # outside the rows
    want = 3.0 / (np.sqrt(2 * 3 * 3 * 4.0) + 1e-8)
    assert orp.deviation(eps, ref, (1, 4)) == pytest.approx(want, rel=1e-15)


def test_unbounded_tolerance_freezes_everything_at_step_two():
    cfg, w, x = load("tiny_ragged")
    r = orp.search(om.Model(cfg, w, x), x["z"], tau_agree=1e30)
    assert r.lifetimes.tolist() == [1] * cfg.L
    assert [s for s, _ in r.order] == [2] * cfg.L


def test_zero_tolerance_freezes_exactly_the_inert_units():
    """tau = 0 admits only candidates whose freezing leaves the output bit for bit the same:
    the units whose branches are identically zero; ties (two inert units, both at deviation
    0) go to the lower index first."""
    cfg, w, x = load("tiny_ragged")
    m = om.Model(cfg, zero_units(w, [0, 2]), x)
    r = orp.search(m, x["z"], tau_agree=0.0)
    assert r.lifetimes.tolist() == [1, cfg.T, 1]
    assert r.order == [(2, 0), (2, 2)]
    assert r.log[(2, 0, 0)] == 0.0 and r.log[(2, 0, 2)] == 0.0 and r.log[(2, 0, 1)] > 0.0


def test_ceiling_forces_least_deviation_units():
    """With tau = 0 and a ceiling of 12 of 18 layer-steps, step 2 must freeze two units (3 +
    5 x 2 = 13 > 12 >= 3 + 5 x 1): the two of least single-unit deviation, which this test
    measures itself by freezing each unit alone at step 2 of the unscheduled trajectory."""
    cfg, w, x = load("tiny_ragged")
    m = om.Model(cfg, w, x)
    r = orp.search(m, x["z"], tau_agree=0.0, max_layer_steps=12)
    # independent check of the first choice
    ups = {}
    ref1 = om.denoise_step(m, x["z"], 1, [1] * cfg.L, ups)
    z2 = om.sampler_update(cfg, np.asarray(x["z"], np.float64), ref1, 1)
    ref2 = om.denoise_step(m, z2, 2, [1] * cfg.L, {})
    single = []
    for j in range(cfg.L):
        row = [0 if l == j else 1 for l in range(cfg.L)]
        e = om.denoise_step(m, z2, 2, row, dict(ups))
        single.append(orp.deviation(e, ref2, cfg.update_rows))
    first = int(np.argmin(single))
    assert r.order[0] == (2, first)
    assert r.log[(2, 0, first)] == single[first]
    assert len([o for o in r.order if o[0] == 2]) == 2
    assert sorted(r.lifetimes.tolist()).count(1) == 2
    active_layer_steps = sum(int(np.sum(np.arange(1, cfg.T + 1) <= S)) for S in r.lifetimes)
    assert active_layer_steps <= 12


def test_replay_of_the_found_schedule_meets_the_tolerance_at_step_two():
    """The pattern found at step 2 keeps the deviation within tau there."""
    cfg, w, x = load("llada_mini")
    m = om.Model(cfg, w, x)
    tau = 5e-3
    r = orp.search(m, x["z"], tau_agree=tau)
    frozen2 = [l for s, l in r.order if s == 2]
    if frozen2:
        assert r.log[(2, len(frozen2) - 1, frozen2[-1])] <= tau
    assert r.evaluations >= cfg.T
