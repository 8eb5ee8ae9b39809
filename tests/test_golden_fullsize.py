"""Consistency of the stored full-size oracle statistics (tests/golden/fullsize_*.txt),
which the GPU schedule tests compare against: the stored unit scores follow from the stored
matrix scores by the block equations, the energies satisfy the identities the paper's
definitions imply, and every schedule built from them lies far from a tie."""
import numpy as np
import pytest

import synth
from oracle import rules as ru
from oracle import schedule as osch
from oracle import spectral as osp

from helpers import load_fullsize_golden

NAMES = ["tiny", "dit", "uvit", "sdxl", "llada", "sdxl_unet"]


@pytest.mark.parametrize("name", NAMES)
def test_golden_consistent(name):
    cfg = synth.get_config(name)
    stats, raw = load_fullsize_golden(name)
    assert len(stats) == len(raw) == cfg.L
    want = {"q", "k", "v", "o", "w1", "w2"} | ({"xq", "xk", "xv", "xo"} if cfg.arch in ("sdxl", "sdxl_unet") else set())
    want |= {"conv1", "conv2"} if cfg.arch == "sdxl_unet" else set()
    for u in stats:
        assert set(u) == want
        for st in u.values():
            # the eigenvalues of the Gram matrix sum to its trace ||W||_F^2
            assert st.energy_top + st.energy_tail == pytest.approx(st.frob_sq, rel=1e-9)
            # the largest of the top-k squared singular values is at least their mean
            assert st.sigma1_sq * st.k >= st.energy_top * (1 - 1e-12)
            assert st.sigma1_sq <= st.energy_top * (1 + 1e-12)
    assert np.allclose(ru.raw_scores("scr_frob", stats, cfg.dh), raw, rtol=1e-14, atol=0)


@pytest.mark.parametrize("name", NAMES)
def test_golden_schedules_far_from_ties(name):
    cfg = synth.get_config(name)
    stats, _ = load_fullsize_golden(name)
    for rule in ru.RULES:
        lam = osp.normalise(ru.raw_scores(rule, stats, cfg.dh, seed=5, L=cfg.L))
        for pct in cfg.budgets:
            n = osch.budget_layer_steps(pct, cfg.L, cfg.T)
            bs = osch.lifetimes_budget(lam, cfg.T, n, osch.s_min_default(cfg.T))
            if rule not in ("depth", "random"):  # exact scores: ties are resolved identically
                assert bs.cut_margin > 1e-8, (rule, pct, bs.cut_margin)
