"""Pins for the static ranking rules of the oracle (Sec. "Static ranking comparisons",
Table "Static rankings at matched layer-step budgets")."""
import math

import numpy as np
import pytest

import functools

import synth
from oracle import rules as ru
from oracle import schedule as sch
from oracle import spectral as sp


def test_splitmix64_known_answers():
    """Published reference outputs of SplitMix64 for seed 1234567 (the first five)."""
    want = [6457827717110365317, 3203168211198807973, 9817491932198370423, 4593380528125082431,
            16408922859458223821]
    assert [ru.splitmix64(1234567, i) for i in range(1, 6)] == want


def test_random_raw_in_unit_interval_and_seeded():
    a = ru.random_raw(50, 7)
    assert np.all((a >= 0) & (a < 1))
    assert np.array_equal(a, ru.random_raw(50, 7))
    assert not np.array_equal(a, ru.random_raw(50, 8))
    b = ru.random_raw(3, 1234567)
    assert b[0] == (6457827717110365317 >> 11) * 2.0 ** -53


def _diag(s, m=None, n=None):
    s = np.asarray(s, np.float64)
    m = m or len(s)
    n = n or len(s)
    w = np.zeros((m, n))
    w[np.arange(len(s)), np.arange(len(s))] = s
    return w


def test_matrix_statistics_closed_forms():
    s = np.array([5.0, 2.0, 1.0, 1.0, 0.5, 0.25, 0.25, 0.1, 0.1, 0.05, 0.01])  # d = 11 -> k = 1
    st = sp.matrix_stats(_diag(s, 13, 11), eta=0.0)
    F = float(np.sum(s * s))
    assert st.sigma1_sq == pytest.approx(25.0, rel=1e-14)
    assert ru.statistic(st, "frob") == pytest.approx(math.sqrt(F), rel=1e-14)
    assert ru.statistic(st, "spectral") == pytest.approx(5.0, rel=1e-14)
    assert ru.statistic(st, "stable_rank") == pytest.approx(25.0 / F, rel=1e-14)
    assert ru.statistic(st, "frob_srank") == pytest.approx(25.0 / math.sqrt(F), rel=1e-14)
    # k = 1, eta = 0: rho = sigma_1^2 / F, so raw SCR = sqrt(rho) and g = ||W||_F sqrt(rho) = sigma_1
    assert ru.statistic(st, "raw_scr") == pytest.approx(math.sqrt(25.0 / F), rel=1e-14)
    assert ru.statistic(st, "scr_frob") == pytest.approx(5.0, rel=1e-14)


@pytest.mark.parametrize("seed", range(6))
def test_sigma1_two_by_two_analytic(seed):
    """||W||_2^2 of a 2 x 2 matrix: the larger root of x^2 - S x + det^2 = 0, S = ||W||_F^2."""
    a, b, c, d = np.random.default_rng(seed).standard_normal(4)
    S = a * a + b * b + c * c + d * d
    det = a * d - b * c
    want = (S + math.sqrt(S * S - 4 * det * det)) / 2
    st = sp.matrix_stats(np.array([[a, b], [c, d]]), eta=0.0)
    assert st.sigma1_sq == pytest.approx(want, rel=1e-13)


def test_sigma1_of_planted_matrices():
    """The generator plants the singular values; the largest one comes back as ||W||_2,
    through the SVD branch (d <= 1024) and the Gram branch (d > 1024)."""
    rng = np.random.default_rng(5)
    for m, n in ((300, 200), (1100, 1030)):
        w, p = synth.planted_matrix(rng, m, n, np.float64)
        st = sp.matrix_stats(w, eta=0.0)
        assert st.sigma1_sq == pytest.approx(p.s[0] ** 2, rel=1e-10)


def _unit(scale_q, spec):
    """A 12 x 12 unit: every matrix is scale * diag(spec)."""
    w = _diag(np.asarray(spec) * scale_q)
    return {r: sp.matrix_stats(w, eta=1e-6) for r in ("q", "k", "v", "o", "w1", "w2")}


def test_rule_orders_on_crafted_spectra():
    """Unit 0: a flat spectrum of large norm.  Unit 1: one dominant direction, smaller
    norm.  Unit 2: unit 1's spectrum at twice the scale.
    Frobenius and spectral norm rank by magnitude; the oriented stable rank and raw SCR are
    scale-free and prefer the concentrated spectra; depth prefers the deepest unit."""
    flat = np.ones(12)
    peak = np.array([3.0] + [0.1] * 11)
    units = [_unit(1.0, flat), _unit(1.0, peak), _unit(2.0, peak)]
    F_flat, F_peak = 12.0, 9.0 + 11 * 0.01
    dh = 4

    def q(gamma):  # block formula with one gamma for all six matrices
        return gamma * gamma * (1 + gamma * gamma / math.sqrt(dh)) + gamma * gamma

    got = {r: ru.raw_scores(r, units, dh) for r in ru.MATRIX_RULES}
    assert got["frob"] == pytest.approx([q(math.sqrt(F_flat)), q(math.sqrt(F_peak)), q(2 * math.sqrt(F_peak))],
                                        rel=1e-12)
    assert got["spectral"] == pytest.approx([q(1.0), q(3.0), q(6.0)], rel=1e-12)
    sr_flat, sr_peak = 1.0 / 12.0, 9.0 / F_peak
    assert got["stable_rank"] == pytest.approx([q(sr_flat), q(sr_peak), q(sr_peak)], rel=1e-12)
    assert got["stable_rank"][1] == got["stable_rank"][2]  # scale-free
    assert got["raw_scr"][1] == pytest.approx(got["raw_scr"][2], rel=1e-12)
    assert np.argsort(got["frob"]).tolist() == [1, 0, 2]
    assert np.argsort(got["spectral"]).tolist() == [0, 1, 2]
    assert got["stable_rank"][0] < got["stable_rank"][1]
    assert got["raw_scr"][0] < got["raw_scr"][1]
    # the method is the Frobenius rule's gamma times the raw-SCR rule's gamma, matrix by matrix
    for u in units:
        for st in u.values():
            assert ru.statistic(st, "scr_frob") == pytest.approx(
                ru.statistic(st, "frob") * ru.statistic(st, "raw_scr"), rel=1e-14)
    d = ru.raw_scores("depth", [], dh, L=3)
    assert d.tolist() == [1.0, 2.0, 3.0]


def test_method_rule_matches_unit_score():
    cfg = synth.get_config("tiny_ragged")
    w = synth.model_weights(cfg)
    stats = [sp.unit_score(sp.unit_matrices(u, cfg.d, cfg.dtype), cfg.dh).stats for u in w]
    raw = ru.raw_scores("scr_frob", stats, cfg.dh)
    ref = [sp.unit_score(sp.unit_matrices(u, cfg.d, cfg.dtype), cfg.dh).raw for u in w]
    assert raw.tolist() == ref


@functools.lru_cache(maxsize=None)
def _mini_stats(name):
    cfg = synth.get_config(name)
    w = synth.model_weights(cfg)
    return cfg, [sp.unit_score(sp.unit_matrices(u, cfg.d, cfg.dtype), cfg.dh).stats for u in w]


@pytest.mark.parametrize("rule", ru.RULES)
def test_every_rule_meets_the_budget(rule):
    cfg, stats = _mini_stats("llada_mini")
    T, L = cfg.T, cfg.L
    for pct in cfg.budgets:
        n = sch.budget_layer_steps(pct, L, T)
        bs = ru.lifetimes(rule, stats, cfg.dh, T, n, sch.s_min_default(T), seed=3)
        assert int(bs.lifetimes.sum()) == n
        assert bs.lifetimes.min() >= sch.s_min_default(T) and bs.lifetimes.max() <= T
    if rule == "depth":
        n = sch.budget_layer_steps(50, L, T)
        S = ru.lifetimes("depth", [], cfg.dh, T, n, sch.s_min_default(T), L=L).lifetimes
        assert np.all(np.diff(S) >= 0)  # deeper units never die earlier
